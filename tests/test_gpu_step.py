"""GPU parity of the fused decode step (dfssm_mamba2_decode_step at one
token on a prepared workspace: all layers in one persistent launch) against
the oracle, against the per-kernel step, under graph capture, and on an
unprepared workspace (which takes the per-kernel sequence).

Every stage follows the oracle's rounding order except the two fp64 sums
(a norm's sum of squares, the SSM's sum over the state), which the device
takes in another order: a result can move by one ulp when an fp64 sum lies
on a rounding boundary, and then, rarely, a code.  So logits must agree
within 1e-3 of their largest value, with the same argmax, and the tests
report how many tokens are bit-exact (in practice all)."""
import numpy as np
import pytest

import dfssm_synth as S
import oracle
from gpu_util import dev, forced_switch, host, say, torch_cuda
from test_gpu_model import EPS, OracleModel, V, _logits_check, device_model

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch = torch_cuda()
    import paper_2606_10932_amd as D
    oracle.build()
    return torch, D, oracle.get()


@pytest.fixture(scope="module")
def model3():
    """Three layers of the 1.3B shapes (r = 64 in every projection but the
    middle layer's, which has r = 12 and r = 0), a 1,000-word table."""
    ws = S.sweep_weights(n_layers=3)
    layers = []
    for l in range(3):
        p = S.mamba_params(2048, key=(160, l))
        ip, op = ws[2 * l], ws[2 * l + 1]
        if l == 1:
            ip = S.weights(2048, 8512, 12, key=(161, 0))
            op = S.weights(4096, 2048, 0, key=(161, 1))
        layers.append(dict(p, in_proj=ip, out_proj=op))
    E, scale = S.embedding(V, 2048, key=(162,))
    norm_f = np.random.default_rng(163).uniform(0.8, 1.2, 2048).astype(np.float32)
    return dict(E=E, scale=scale, norm_f=norm_f, layers=layers)


def test_fused_step_against_oracle_and_per_kernel(env, model3, record_property):
    torch, D, o = env
    T = 6
    say(f"fused decode step, 3 layers, M=1, {T} tokens: oracle and the per-kernel step")
    m = device_model(D, model3)
    ring, state = m.new_state(1)
    ws = m.workspace(1)
    ring_k, state_k = m.new_state(1)
    ws_k = m.workspace(1)
    assert m.fused_path(1, ws) and m.fused_path(1, ws_k)
    with forced_switch(D, D.TEST_STEP_PER_KERNEL, 1):
        assert not m.fused_path(1, ws)
    om = OracleModel(o, model3, 1)
    exact = same = 0
    for t in range(T):
        tok = S.tokens(1, V, key=(164, t))
        lg = host(m.decode_step(dev(tok), t, ring, state, ws))
        with forced_switch(D, D.TEST_STEP_PER_KERNEL, 1):
            lk = host(m.decode_step(dev(tok), t, ring_k, state_k, ws_k))
        torch.cuda.synchronize()
        st = m.status(1, ws)
        assert st == 0, f"token {t}: status word {st:#x} (bits {st & 0xffff:#x}, linear {(st >> 16) - 1})"
        ref = om.step(tok)
        exact += _logits_check(lg, ref, f"fused, token {t}")
        _logits_check(lk, ref, f"per-kernel, token {t}")
        same += int(np.array_equal(lg.view(np.uint32), lk.view(np.uint32)))
    # the state after T tokens: the same values as the oracle's to the fp64
    # sums' rounding
    for l in range(3):
        st = host(state).reshape(3, 64, 64, 128)[l]
        ref_st = om.ssm[l][0]
        assert np.abs(st - ref_st).max() <= 1e-5 * max(1.0, float(np.abs(ref_st).max())), f"layer {l} state"
    say(f"  {exact} of {T} tokens bit-exact against the oracle, {same} against the per-kernel step")
    record_property("bit_exact_tokens", f"{exact}/{T}")
    assert exact >= T - 1


def test_fused_step_graph_replays(env, model3, record_property):
    """Four captured fused steps (one per ring slot) replayed token after
    token with new token ids between replays: every replay equals the eager
    fused step bit for bit and the oracle within the bar."""
    torch, D, o = env
    T = 8
    say(f"fused decode step: four captured graphs, {T} replays at M=1")
    m = device_model(D, model3)
    ring_e, state_e = m.new_state(1)
    ws_e = m.workspace(1)
    toks = [S.tokens(1, V, key=(165, t)) for t in range(T)]
    eager = [host(m.decode_step(dev(tk), t, ring_e, state_e, ws_e)) for t, tk in enumerate(toks)]
    torch.cuda.synchronize()
    assert m.status(1, ws_e) == 0
    ring, state = m.new_state(1)
    ws = m.workspace(1)
    tok_buf = torch.zeros(1, dtype=torch.int32, device="cuda")
    lg_buf = torch.empty((1, V), dtype=torch.float32, device="cuda")
    ring_c, state_c = m.new_state(1)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graphs = []
    with torch.cuda.stream(side):
        m.decode_step(tok_buf, 0, ring_c, state_c, ws, logits=lg_buf)
        for ph in range(4):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                m.decode_step(tok_buf, ph, ring, state, ws, logits=lg_buf)
            graphs.append(g)
    torch.cuda.synchronize()
    ring.zero_()
    state.zero_()
    torch.cuda.synchronize()
    om = OracleModel(o, model3, 1)
    exact = 0
    for t, tk in enumerate(toks):
        tok_buf.copy_(dev(tk))
        torch.cuda.synchronize()
        graphs[t % 4].replay()
        torch.cuda.synchronize()
        got = host(lg_buf)
        assert np.array_equal(got.view(np.uint32), eager[t].view(np.uint32)), f"replay for token {t}"
        exact += _logits_check(got, om.step(tk), f"replay for token {t} against the oracle")
    assert m.status(1, ws) == 0
    assert np.array_equal(host(state), host(state_e)) and np.array_equal(host(ring), host(ring_e))
    say(f"  {exact} of {T} replays bit-exact against the oracle")
    record_property("bit_exact_tokens", f"{exact}/{T}")


def test_unprepared_workspace_runs_per_kernel(env, model3):
    """Without dfssm_mamba2_prepare the step at M = 1 takes the per-kernel
    sequence (the same logits as the fused step on the same inputs, within
    the bar) and the status query reports 0."""
    torch, D, o = env
    say("decode step on an unprepared workspace")
    m = device_model(D, model3)
    ring, state = m.new_state(1)
    ws = m.workspace(1, prepare=False)
    assert not m.fused_path(1, ws)
    om = OracleModel(o, model3, 1)
    for t in range(2):
        tok = S.tokens(1, V, key=(166, t))
        lg = host(m.decode_step(dev(tok), t, ring, state, ws))
        torch.cuda.synchronize()
        _logits_check(lg, om.step(tok), f"token {t}")
    assert m.status(1, ws) == 0


def _tie_model(model3):
    """model3 with layer 0's norm weights all 1 and embedding rows whose
    largest entries tie: row 7 constant (every entry ties), row 8 two
    largest entries in one lane's eight (3 and 5), row 9 two in different
    lanes (3 and 17), row 10 all zero."""
    md = dict(model3)
    E = model3["E"].copy()
    E[7] = 40
    for row, ids in ((8, (3, 5)), (9, (3, 17))):
        E[row] = np.clip(E[row], -60, 60)
        E[row, list(ids)] = 100
    E[10] = 0
    md["E"] = E
    md["layers"] = [dict(model3["layers"][0], norm_w=np.ones(2048, np.float32))] + list(model3["layers"][1:])
    return md


@pytest.mark.parametrize("tied", [False, True])
def test_fused_step_one_and_two_exchanges(env, model3, tied, record_property):
    """The input maxima from one exchange (the published largest entries)
    and from the second exchange (forced) give the same bits, both within
    the bar of the oracle; with tied largest entries (every entry of a
    constant row ties, which takes the second exchange) and a zero row."""
    torch, D, o = env
    md = _tie_model(model3) if tied else model3
    toks = [np.array([t], np.int32) for t in (7, 8, 9, 10, 7)] if tied else \
        [S.tokens(1, V, key=(167, t)) for t in range(4)]
    say(f"fused decode step: one and two exchanges for the input maxima, {'tied' if tied else 'random'} tokens")
    m = device_model(D, md)
    ring, state = m.new_state(1)
    ws = m.workspace(1)
    ring2, state2 = m.new_state(1)
    ws2 = m.workspace(1)
    om = OracleModel(o, md, 1)
    exact = 0
    for t, tk in enumerate(toks):
        lg = host(m.decode_step(dev(tk), t, ring, state, ws))
        with forced_switch(D, D.TEST_STEP_PER_KERNEL, 2):
            l2 = host(m.decode_step(dev(tk), t, ring2, state2, ws2))
        torch.cuda.synchronize()
        assert m.status(1, ws) == 0 and m.status(1, ws2) == 0
        assert np.array_equal(lg.view(np.uint32), l2.view(np.uint32)), f"token {t}: one and two exchanges differ"
        exact += _logits_check(lg, om.step(tk), f"token {t}")
    assert np.array_equal(host(state), host(state2))
    say(f"  {exact} of {len(toks)} tokens bit-exact against the oracle")
    record_property("bit_exact_tokens", f"{exact}/{len(toks)}")


def test_fused_step_int4_lora(env, model3, record_property):
    """The fused step with int4 LoRA factors (Table 4) in every projection
    (r = 64, 8 and 16): against the oracle and the per-kernel step."""
    torch, D, o = env
    T = 4
    md = dict(model3)
    md["layers"] = [dict({k: v for k, v in ly.items() if k not in ("in_proj", "out_proj")},
                         in_proj=S.weights_i4(2048, 8512, (64, 8, 16)[l], key=(168, l, 0)),
                         out_proj=S.weights_i4(4096, 2048, (64, 16, 8)[l], key=(168, l, 1)))
                    for l, ly in enumerate(model3["layers"])]
    say(f"fused decode step with int4 LoRA, 3 layers, M=1, {T} tokens")
    m = device_model(D, md)
    ring, state = m.new_state(1)
    ws = m.workspace(1)
    ring_k, state_k = m.new_state(1)
    ws_k = m.workspace(1)
    assert m.fused_path(1, ws)
    om = OracleModel(o, md, 1)
    exact = same = 0
    for t in range(T):
        tok = S.tokens(1, V, key=(169, t))
        lg = host(m.decode_step(dev(tok), t, ring, state, ws))
        with forced_switch(D, D.TEST_STEP_PER_KERNEL, 1):
            lk = host(m.decode_step(dev(tok), t, ring_k, state_k, ws_k))
        torch.cuda.synchronize()
        assert m.status(1, ws) == 0
        exact += _logits_check(lg, om.step(tok), f"fused int4, token {t}")
        same += int(np.array_equal(lg.view(np.uint32), lk.view(np.uint32)))
    say(f"  {exact} of {T} tokens bit-exact against the oracle, {same} against the per-kernel step")
    record_property("bit_exact_tokens", f"{exact}/{T}")
    assert exact >= T - 1
