"""GPU parity of the whole decode step (dfssm_mamba2_decode_step): token
gather, every layer's norm -> in_proj -> conv + SSM step -> gated norm ->
out_proj with the residual, final norm and LM head, over several tokens.

Against the oracle: the same chain of oracle calls on the same seeded model
(the 1.3B layer shapes, 2 layers, a 1,000-word table), with int8 LoRA
factors, and again with int4 ones.  Every stage follows
one rounding order; the SSM output's fp64 sum is taken in another order on
the device, which can move a value by one ulp and, rarely, a code of
out_proj's input, so logits must agree within 1e-3 of their largest value
(and the argmax must agree), and in practice agree bit for bit.

Against itself and the oracle under graph capture: four captured steps
(one per ring slot, step & 3) replayed token after token, with new token
ids written between replays, must give exactly the eager results, replay
after replay, and the oracle's within the same bar (at 2 sequences, and at
130, where in_proj takes the prefill path).

At the full size: the 48-layer 1.3B model with its 50,280-word table at
batch 1 and 8 over 4 tokens against the oracle, reporting how many tokens'
logits are bit-exact."""
import numpy as np
import pytest

import dfssm_synth as S
import oracle
from gpu_util import dev, dev_weights, host, say, torch_cuda

pytestmark = pytest.mark.gpu

V, L, EPS = 1000, 2, 1e-5


@pytest.fixture(scope="module")
def env():
    torch = torch_cuda()
    import paper_2606_10932_amd as D
    oracle.build()
    return torch, D, oracle.get()


@pytest.fixture(scope="module")
def model_host():
    ws = S.sweep_weights(n_layers=L)
    layers = []
    for l in range(L):
        p = S.mamba_params(2048, key=(140, l))
        layers.append(dict(p, in_proj=ws[2 * l], out_proj=ws[2 * l + 1]))
    E, scale = S.embedding(V, 2048, key=(141,))
    norm_f = np.random.default_rng(142).uniform(0.8, 1.2, 2048).astype(np.float32)
    return dict(E=E, scale=scale, norm_f=norm_f, layers=layers)


@pytest.fixture(scope="module")
def model_host_i4():
    # the same model with int4 LoRA factors (r = 64) in every projection
    layers = []
    for l in range(L):
        p = S.mamba_params(2048, key=(145, l))
        layers.append(dict(p, in_proj=S.weights_i4(2048, 8512, 64, key=(146, l, 0)),
                           out_proj=S.weights_i4(4096, 2048, 64, key=(146, l, 1))))
    E, scale = S.embedding(V, 2048, key=(147,))
    norm_f = np.random.default_rng(148).uniform(0.8, 1.2, 2048).astype(np.float32)
    return dict(E=E, scale=scale, norm_f=norm_f, layers=layers)


def device_model(D, mh):
    layers = []
    for ly in mh["layers"]:
        d = {k: dev(v) for k, v in ly.items() if k not in ("in_proj", "out_proj")}
        for pj in ("in_proj", "out_proj"):
            d[pj] = {k: dev(v) for k, v in ly[pj].items()} if "A4" in ly[pj] else dev_weights(ly[pj])
        layers.append(d)
    return D.Mamba2(dev(mh["E"]), dev(mh["scale"]), dev(mh["norm_f"]), layers, d_state=128, eps=EPS)


class OracleModel:
    """The decode step as a sequence of oracle calls (test-side plumbing)."""

    def __init__(self, o, mh, M):
        self.o, self.mh, self.M = o, mh, M
        dm = S.mamba_dims(2048)
        n = len(mh["layers"])
        self.conv = [np.zeros((M, dm["conv_dim"], 4), np.float32) for _ in range(n)]
        self.ssm = [np.zeros((M, 64, 64, 128), np.float32) for _ in range(n)]

    def _linear(self, q, s, w):
        return (self.o.linear_i4(q, s, **w) if "A4" in w else self.o.linear(q, s, **w))["y32"]

    def step(self, tok):
        o, mh = self.o, self.mh
        u = o.embed_gather(mh["E"], mh["scale"], tok)
        delta = None
        for l, ly in enumerate(mh["layers"]):
            u, _, q, s = o.add_rmsnorm_quant(u, ly["norm_w"], EPS, delta=delta)
            zx = self._linear(q, s, ly["in_proj"])
            y, _, self.conv[l], self.ssm[l] = o.ssm_step(zx, self.conv[l], self.ssm[l], ly["conv_w"], ly["conv_b"],
                                                         ly["dt_bias"], ly["A_log"], ly["D"], 4096, 128, 64)
            _, q, s = o.gate_norm_quant(y, zx[:, :4096], ly["gate_w"], EPS)
            delta = self._linear(q, s, ly["out_proj"])
        _, _, q, s = o.add_rmsnorm_quant(u, mh["norm_f"], EPS, delta=delta)
        return o.lm_head(q, s, mh["E"], mh["scale"])[1]


@pytest.mark.parametrize("M", [1, 3])
def test_decode_step_against_oracle(env, model_host, M):
    torch, D, o = env
    say(f"decode step M={M} vs oracle")
    m = device_model(D, model_host)
    ring, state = m.new_state(M)
    ws = m.workspace(M)
    om = OracleModel(o, model_host, M)
    exact = 0
    for t in range(5):
        tok = S.tokens(M, V, key=(143, M, t))
        ref = om.step(tok)
        lg = host(m.decode_step(dev(tok), t, ring, state, ws))
        torch.cuda.synchronize()
        scale = float(np.abs(ref).max())
        assert np.abs(lg.astype(np.float64) - ref).max() <= 1e-3 * scale, f"token {t}"
        assert np.array_equal(lg.argmax(axis=1), ref.argmax(axis=1)), f"token {t}"
        exact += int(np.array_equal(lg.view(np.uint32), ref.view(np.uint32)))
    say(f"  {exact} of 5 tokens bit-exact")
    assert exact >= 3


@pytest.mark.parametrize("M,steps", [(2, 4), (130, 1)])
def test_decode_step_int4_lora(env, model_host_i4, M, steps):
    # int4 factors in every projection: the few-token kernel reads them
    # packed (both projections at M = 2, out_proj at M = 130); in_proj at
    # M = 130 takes the prefill path on factors expanded in the workspace
    torch, D, o = env
    say(f"decode step, int4 LoRA, M={M} vs oracle")
    m = device_model(D, model_host_i4)
    ring, state = m.new_state(M)
    ws = m.workspace(M)
    om = OracleModel(o, model_host_i4, M)
    exact = 0
    for t in range(steps):
        tok = S.tokens(M, V, key=(149, M, t))
        ref = om.step(tok)
        lg = host(m.decode_step(dev(tok), t, ring, state, ws))
        torch.cuda.synchronize()
        scale = float(np.abs(ref).max())
        assert np.abs(lg.astype(np.float64) - ref).max() <= 1e-3 * scale, f"token {t}"
        assert np.array_equal(lg.argmax(axis=1), ref.argmax(axis=1)), f"token {t}"
        exact += int(np.array_equal(lg.view(np.uint32), ref.view(np.uint32)))
    say(f"  {exact} of {steps} tokens bit-exact")


def _logits_check(lg, ref, what):
    scale = float(np.abs(ref).max())
    assert np.abs(lg.astype(np.float64) - ref).max() <= 1e-3 * scale, what
    assert np.array_equal(lg.argmax(axis=1), ref.argmax(axis=1)), what
    return int(np.array_equal(lg.view(np.uint32), ref.view(np.uint32)))


@pytest.mark.parametrize("M,T", [(2, 8), (130, 4)])
def test_decode_step_graph_replays(env, model_host, M, T, record_property):
    torch, D, o = env
    say(f"decode step: four captured graphs, {T} replays at M={M}, against eager and the oracle")
    m = device_model(D, model_host)
    # eager reference on its own state
    ring_e, state_e = m.new_state(M)
    ws_e = m.workspace(M)
    toks = [S.tokens(M, V, key=(144, M, t)) for t in range(T)]
    eager = [host(m.decode_step(dev(tk), t, ring_e, state_e, ws_e)) for t, tk in enumerate(toks)]
    torch.cuda.synchronize()
    # graphs: static token buffer, logits buffer and workspace
    ring, state = m.new_state(M)
    ws = m.workspace(M)
    tok_buf = torch.zeros(M, dtype=torch.int32, device="cuda")
    lg_buf = torch.empty((M, V), dtype=torch.float32, device="cuda")
    # capture on scratch state so the real state stays at token 0
    ring_c, state_c = m.new_state(M)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graphs = []
    with torch.cuda.stream(side):
        m.decode_step(tok_buf, 0, ring_c, state_c, ws, logits=lg_buf)     # warm-up outside capture
        for ph in range(4):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                m.decode_step(tok_buf, ph, ring, state, ws, logits=lg_buf)
            graphs.append(g)
    torch.cuda.synchronize()
    # the captures did not run: reset the state the graphs write
    ring.zero_()
    state.zero_()
    torch.cuda.synchronize()
    om = OracleModel(o, model_host, M)
    exact = 0
    for t, tk in enumerate(toks):
        tok_buf.copy_(dev(tk))
        torch.cuda.synchronize()
        graphs[t % 4].replay()
        torch.cuda.synchronize()
        got = host(lg_buf)
        assert np.array_equal(got.view(np.uint32), eager[t].view(np.uint32)), f"replay for token {t}"
        exact += _logits_check(got, om.step(tk), f"replay for token {t} against the oracle")
    assert np.array_equal(host(state), host(state_e)) and np.array_equal(host(ring), host(ring_e))
    say(f"  {exact} of {T} replays bit-exact against the oracle")
    record_property("bit_exact_tokens", f"{exact}/{T}")


@pytest.fixture(scope="module")
def model_host_full():
    """The 1.3B model: 48 layers of the sweep's seeded projections, seeded
    layer parameters, the 50,280 x 2048 tied table."""
    ws = S.sweep_weights(n_layers=48)
    layers = []
    for l in range(48):
        p = S.mamba_params(2048, key=(150, l))
        layers.append(dict(p, in_proj=ws[2 * l], out_proj=ws[2 * l + 1]))
    E, scale = S.embedding(50280, 2048, key=(151,))
    norm_f = np.random.default_rng(152).uniform(0.8, 1.2, 2048).astype(np.float32)
    return dict(E=E, scale=scale, norm_f=norm_f, layers=layers)


@pytest.mark.parametrize("M", [1, 8])
def test_decode_step_full_model(env, model_host_full, M, record_property):
    torch, D, o = env
    T = 4
    say(f"decode step: 48-layer 1.3B model, batch {M}, {T} tokens vs oracle")
    m = device_model(D, model_host_full)
    ring, state = m.new_state(M)
    ws = m.workspace(M)
    assert m.fused_path(M, ws) == (M == 1)   # batch 1: one persistent launch for the 48 layers
    om = OracleModel(o, model_host_full, M)
    exact = 0
    for t in range(T):
        tok = S.tokens(M, 50280, key=(153, M, t))
        lg = host(m.decode_step(dev(tok), t, ring, state, ws))
        torch.cuda.synchronize()
        exact += _logits_check(lg, om.step(tok), f"token {t}")
    assert m.status(M, ws) == 0
    say(f"  {exact} of {T} tokens bit-exact against the oracle" + (" (the fused step)" if M == 1 else ""))
    record_property("bit_exact_tokens", f"{exact}/{T}")
