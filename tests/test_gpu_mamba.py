"""GPU parity of the Mamba-2 decode step around the linears, through the C
ABI, against the CPU oracle on the same seeded inputs: residual RMSNorm +
quantisation, the convolution + SSM step over several tokens, gate-then-norm
+ quantisation, and one whole decode layer with the two linears.

Both sides follow one pinned rounding order (fp32 elementwise, fp64
transcendentals and reductions rounded once), so the int8 codes, the scales,
the residual sums and the states must match bit for bit.  The SSM output y
is a 128-term fp64 sum taken in another order on the device; it must match
to one fp32 ulp (and does bit for bit unless a sum sits on a rounding
boundary).  Shapes are the 1.3B model's (d_model 2048, d_inner 4096, 64
heads of 64, d_state 128) plus a d_state 64 variant and ragged sizes."""
import numpy as np
import pytest

import dfssm_synth as S
import oracle
from gpu_util import dev, dev_weights, host, say, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch = torch_cuda()
    import paper_2606_10932_amd as D
    oracle.build()
    return torch, D, oracle.get()


def to_ring(shift: np.ndarray, t: int) -> np.ndarray:
    """Shift register [M, C, 4] (position 3 newest) before step t -> the
    library's ring [M, 4, C]: position j is slot (t - 4 + j) & 3."""
    M, C, _ = shift.shape
    ring = np.zeros((M, 4, C), np.float32)
    for j in range(4):
        ring[:, (t - 4 + j) % 4, :] = shift[:, :, j]
    return ring


def from_ring(ring: np.ndarray, t: int) -> np.ndarray:
    """The ring before step t -> the shift register [M, C, 4]."""
    M, _, C = ring.shape
    shift = np.zeros((M, C, 4), np.float32)
    for j in range(4):
        shift[:, :, j] = ring[:, (t - 4 + j) % 4, :]
    return shift


def eq_bits(a, b):
    return np.array_equal(np.asarray(a).view(np.uint32), np.asarray(b).view(np.uint32))


def within_ulp(g, r):
    g = np.asarray(g, np.float32)
    r = np.asarray(r, np.float32)
    return np.all(np.abs(g.astype(np.float64) - r) <= np.spacing(np.abs(r)).astype(np.float64))


# ---------------------------------------------------------------- norms
NSHAPES = [(1, 2048), (4, 2048), (3, 4096), (2, 64), (5, 16384), (1, 4), (7, 1028)]


@pytest.mark.parametrize("M,d", NSHAPES)
@pytest.mark.parametrize("mode", ["plain", "residual", "in_place"])
def test_add_rmsnorm_quant(env, M, d, mode):
    torch, D, o = env
    say(f"add_rmsnorm_quant M={M} d={d} {mode}")
    u = S.residual(M, d, key=(110, M, d))
    delta = None if mode == "plain" else S.residual(M, d, key=(111, M, d)) * np.float32(0.3)
    w = np.random.default_rng(113).uniform(0.8, 1.2, d).astype(np.float32)
    u_ref, _, q_ref, s_ref = o.add_rmsnorm_quant(u, w, 1e-5, delta=delta)
    ud = dev(u)
    u_out = ud if mode == "in_place" else torch.empty_like(ud)
    q, s = D.add_rmsnorm_quant(ud, dev(w), 1e-5, delta=None if delta is None else dev(delta), u_out=u_out)
    torch.cuda.synchronize()
    assert np.array_equal(host(q), q_ref)
    assert eq_bits(host(s), s_ref)
    assert eq_bits(host(u_out), u_ref)


def test_rmsnorm_zero_rows(env):
    torch, D, o = env
    say("add_rmsnorm_quant zero rows")
    u = S.residual(3, 256, key=(114,))
    delta = u.copy()
    delta[1] = -u[1]                       # row 1 sums to zero
    w = np.ones(256, np.float32)
    _, _, q_ref, s_ref = o.add_rmsnorm_quant(u, w, 1e-5, delta=delta)
    q, s = D.add_rmsnorm_quant(dev(u), dev(w), 1e-5, delta=dev(delta))
    torch.cuda.synchronize()
    assert np.array_equal(host(q), q_ref) and eq_bits(host(s), s_ref)
    assert not host(q)[1].any() and host(s)[1] == 0


GSHAPES = [(1, 4096, 8512), (4, 4096, 8512), (3, 2048, 2048), (2, 64, 68), (1, 16384, 16384)]


@pytest.mark.parametrize("M,d,ldz", GSHAPES)
def test_gate_norm_quant(env, M, d, ldz):
    torch, D, o = env
    say(f"gate_norm_quant M={M} d={d} ldz={ldz}")
    y = S.residual(M, d, key=(115, M, d))
    zrow = S.residual(M, ldz, key=(116, M, ldz)) * np.float32(2.0)
    zrow[:, 5:40:3] = 0.0                  # silu(0) = 0: zero channels
    w = np.random.default_rng(117).uniform(0.8, 1.2, d).astype(np.float32)
    _, q_ref, s_ref = o.gate_norm_quant(y, zrow[:, :d], w, 1e-5)
    zd = dev(zrow)
    q, s = D.gate_norm_quant(dev(y), zd[:, :d], dev(w), 1e-5)
    torch.cuda.synchronize()
    assert np.array_equal(host(q), q_ref)
    assert eq_bits(host(s), s_ref)


# ---------------------------------------------------------------- SSM step
def _ssm_run(torch, D, o, M, d_model, N, t0, steps, key):
    dm = S.mamba_dims(d_model, N, 64)
    p = S.mamba_params(d_model, N, 64, key=key)
    st = S.mamba_state(M, d_model, N, 64, key=key)
    cs_ref, hs_ref = st["conv_state"], st["ssm_state"]
    ring = dev(to_ring(cs_ref, t0))
    hs = dev(hs_ref)
    pd = {k: dev(v) for k, v in p.items()}
    for i in range(steps):
        t = t0 + i
        zx = S.inproj_out(M, d_model, N, 64, key=key + (i,))
        y_ref, xbc_ref, cs_ref, hs_ref = o.ssm_step(zx, cs_ref, hs_ref, p["conv_w"], p["conv_b"], p["dt_bias"],
                                                    p["A_log"], p["D"], dm["d_inner"], N, 64)
        xbc = torch.empty((M, dm["conv_dim"]), dtype=torch.float32, device="cuda")
        y = D.ssm_step(dev(zx), t, ring, hs, pd["conv_w"], pd["conv_b"], pd["dt_bias"], pd["A_log"], pd["D"],
                       d_state=N, xbc=xbc)
        torch.cuda.synchronize()
        what = f"M={M} d_model={d_model} N={N} step={t}"
        assert eq_bits(host(xbc), xbc_ref), what + " conv outputs"
        assert eq_bits(from_ring(host(ring), t + 1), cs_ref), what + " conv state"
        assert eq_bits(host(hs), hs_ref), what + " ssm state"
        yg = host(y)
        assert within_ulp(yg, y_ref), what + " y"
        ndiff = int(np.count_nonzero(yg.view(np.uint32) != y_ref.view(np.uint32)))
        assert ndiff <= max(2, yg.size // 10000), what + f" {ndiff} y differ by an ulp"
        # later steps continue from the oracle's state so one ulp cannot grow
        hs.copy_(dev(hs_ref))


SSHAPES = [
    # (M, d_model, d_state, first step, steps)
    (1, 2048, 128, 0, 6),      # the 1.3B mixer, ring wraps
    (3, 2048, 128, 5, 5),
    (8, 2048, 128, 2, 3),
    (2, 1024, 64, 0, 5),       # d_state 64
    (1, 32, 128, 3, 5),        # one head
    (5, 96, 64, 1, 4),         # three heads, ragged M
    (16, 2048, 128, 1, 3),     # 64 channels per workgroup from 16 sequences
    (33, 1024, 64, 0, 2),      # the same with d_state 64
]


@pytest.mark.parametrize("M,d_model,N,t0,steps", SSHAPES)
def test_ssm_step(env, M, d_model, N, t0, steps):
    torch, D, o = env
    say(f"ssm_step M={M} d_model={d_model} N={N} t0={t0}")
    _ssm_run(torch, D, o, M, d_model, N, t0, steps, key=(120, M, d_model, N))


def test_ssm_step_large_step_index(env):
    # the ring position is the step index mod 4, at any size of the index
    torch, D, o = env
    say("ssm_step step index 2^40 + 1")
    _ssm_run(torch, D, o, 2, 256, 128, (1 << 40) + 1, 5, key=(121,))


def test_ssm_step_new_sequence_from_zeros(env):
    # a fresh sequence: zero ring, zero state, first step
    torch, D, o = env
    say("ssm_step from zeros")
    M, dm_ = 2, S.mamba_dims(2048)
    p = S.mamba_params(2048, key=(122,))
    pd = {k: dev(v) for k, v in p.items()}
    cs = np.zeros((M, dm_["conv_dim"], 4), np.float32)
    hs0 = np.zeros((M, 64, 64, 128), np.float32)
    zx = S.inproj_out(M, 2048, key=(122,))
    y_ref, _, cs_ref, hs_ref = o.ssm_step(zx, cs, hs0, p["conv_w"], p["conv_b"], p["dt_bias"], p["A_log"], p["D"],
                                          4096, 128, 64)
    ring = torch.zeros((M, 4, dm_["conv_dim"]), dtype=torch.float32, device="cuda")
    hs = torch.zeros((M, 64, 64, 128), dtype=torch.float32, device="cuda")
    y = D.ssm_step(dev(zx), 0, ring, hs, pd["conv_w"], pd["conv_b"], pd["dt_bias"], pd["A_log"], pd["D"])
    torch.cuda.synchronize()
    assert eq_bits(host(hs), hs_ref) and within_ulp(host(y), y_ref)
    assert eq_bits(from_ring(host(ring), 1), cs_ref)


# ---------------------------------------------------------------- one layer
def test_decode_layer_end_to_end(env):
    """Residual RMSNorm -> in_proj -> conv + SSM step -> gate norm ->
    out_proj -> residual, three tokens in a row of the 1.3B layer shapes, all
    on the device, against the same chain of oracle calls."""
    torch, D, o = env
    say("decode layer end to end")
    M = 2
    dm = S.mamba_dims(2048)
    p = S.mamba_params(2048, key=(130,))
    w_in = S.config_weights(1)
    w_out = S.config_weights(2)
    st = S.mamba_state(M, 2048, key=(130,))
    pd = {k: dev(v) for k, v in p.items()}
    wid, wod = dev_weights(w_in), dev_weights(w_out)
    u_ref = S.residual(M, 2048, key=(130,))
    cs_ref, hs_ref = st["conv_state"], st["ssm_state"]
    ud = dev(u_ref)
    ring = dev(to_ring(cs_ref, 0))
    hs = dev(hs_ref)
    delta_ref, delta = None, None
    for t in range(3):
        # oracle
        u_ref, _, q1, s1 = o.add_rmsnorm_quant(u_ref, p["norm_w"], 1e-5, delta=delta_ref)
        zx = o.linear(q1, s1, **w_in)["y32"]
        y_ssm, _, cs_ref, hs_ref = o.ssm_step(zx, cs_ref, hs_ref, p["conv_w"], p["conv_b"], p["dt_bias"],
                                              p["A_log"], p["D"], 4096, 128, 64)
        _, q2, s2 = o.gate_norm_quant(y_ssm, zx[:, :4096], p["gate_w"], 1e-5)
        delta_ref = o.linear(q2, s2, **w_out)["y32"]
        # device
        qd, sd = D.add_rmsnorm_quant(ud, pd["norm_w"], 1e-5, delta=delta, u_out=ud)
        zxd = D.scaffold_lora_linear(qd, sd, wid["w_bits"], wid["alpha"], wid["A"], wid["B"], wid["beta"])
        yd = D.ssm_step(zxd, t, ring, hs, pd["conv_w"], pd["conv_b"], pd["dt_bias"], pd["A_log"], pd["D"])
        q2d, s2d = D.gate_norm_quant(yd, zxd[:, :4096], pd["gate_w"], 1e-5)
        delta = D.scaffold_lora_linear(q2d, s2d, wod["w_bits"], wod["alpha"], wod["A"], wod["B"], wod["beta"])
        torch.cuda.synchronize()
        what = f"token {t}"
        assert np.array_equal(host(qd), q1) and eq_bits(host(sd), s1), what + " in_proj input"
        assert eq_bits(host(zxd), zx), what + " in_proj output"
        assert within_ulp(host(yd), y_ssm), what + " ssm output"
        g_ok = np.array_equal(host(q2d), q2) and eq_bits(host(s2d), s2)
        if not g_ok:
            # a one-ulp y can move the fp64 sum of squares across a rounding
            # boundary only if y differed; then the codes differ by at most 1
            assert not eq_bits(host(yd), y_ssm), what + " out_proj input differs with equal y"
            assert np.abs(host(q2d).astype(int) - q2).max() <= 1
        else:
            assert eq_bits(host(delta), delta_ref), what + " out_proj output"
        # continue from the oracle's values so both sides see the same input
        ud.copy_(dev(u_ref))
        delta = dev(delta_ref)
        hs.copy_(dev(hs_ref))
        ring.copy_(dev(to_ring(cs_ref, t + 1)))
    assert np.all(np.isfinite(delta_ref))
