"""GPU parity of the tied int8 embedding table: token gather and LM head,
through the C ABI, against the CPU oracle on the same seeded inputs.

acc is exact int32 and must match bit for bit; the logits follow a fixed
fp32 order (s * (scale * (float)acc)) and must match the oracle's fp32
evaluation bit for bit, and the exact product within three roundings.
Both kernels are covered: the GEMV passes (fewer than 8 tokens) and the
matrix-core kernel (from 8 tokens), each also forced through a test switch.
The full-size cases use the 1.3B model's table (50,280 x 2048)."""
import numpy as np
import pytest

import dfssm_synth as S
import oracle
from gpu_util import dev, forced_switch, host, say, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch = torch_cuda()
    import paper_2606_10932_amd as D
    oracle.build()
    return torch, D, oracle.get()


@pytest.fixture(scope="module")
def table_1p3b():
    return S.embedding(S.VOCAB_1P3B, S.D_MODEL_1P3B, key=(40,))


def _table(V, d, key):
    if (V, d) == (S.VOCAB_1P3B, S.D_MODEL_1P3B):
        return None
    return S.embedding(V, d, key=key)


def _check_lm(torch, D, o, q, s, E, scale, what):
    acc_r, lg_r = o.lm_head(q, s, E, scale)
    Ed, sd = dev(E), dev(scale)
    lg, acc = D.lm_head(dev(q), dev(s), Ed, sd, acc=True)
    torch.cuda.synchronize()
    acc_g, lg_g = host(acc), host(lg)
    bad = np.flatnonzero(acc_g != acc_r)
    assert bad.size == 0, f"{what}: {bad.size} acc differ, first {bad[:5]}"
    bad = np.flatnonzero(lg_g.view(np.uint32) != lg_r.view(np.uint32))
    assert bad.size == 0, f"{what}: {bad.size} logits differ from the fp32-ordered oracle, first {bad[:5]}"
    # against the exact product: (float)acc, scale*., s*. are three roundings
    exact = s.astype(np.float64)[:, None] * scale.astype(np.float64)[None, :] * acc_r.astype(np.float64)
    err = np.abs(lg_g.astype(np.float64) - exact)
    assert np.all(err <= 3.001 * 2.0 ** -24 * np.abs(exact)), what


# ---------------------------------------------------------------- LM head
LSHAPES = [
    # (M, d, V)
    (1, 2048, 50280),   # the 1.3B table, one token
    (4, 2048, 50280),   # four tokens: one pass
    (5, 2048, 1001),    # two passes, the second of one token; ragged row groups
    (3, 768, 3001),     # 130M width: 48 of 64 lanes carry codes
    (2, 16, 7),         # one 16-byte slice per row, fewer rows than a visit
    (1, 1040, 333),     # a 1 KB chunk plus a 16-byte tail
    (3, 4112, 130),     # 4 KB chunks + tail: 2 tokens per pass
    (9, 5120, 100),     # 8 KB rows: 2 tokens per pass, 5 passes
    (2, 16384, 65),     # the longest row: 1 token per pass
    # from 8 tokens the matrix-core kernel (d a multiple of 64 split over 4..8 waves)
    (8, 2048, 50280),   # the 1.3B table, the smallest batch it takes
    (17, 1024, 77),
    (40, 4096, 130),    # 8 steps per wave
    # from 64 tokens the tiled kernel (64-token blocks below 128 tokens, 128 from there)
    (64, 2048, 50280),
    (512, 2048, 50280),  # the 1.3B table at the largest decode batch
    (64, 256, 200),     # 4 stages of 64 columns
    (65, 512, 129),     # a second token block of one token; V % 4 != 0
    (130, 1024, 77),    # one partly filled row block
    (300, 768, 1001),   # ragged token and row blocks
]


@pytest.mark.parametrize("M,d,V", LSHAPES)
def test_lm_head(env, table_1p3b, M, d, V):
    torch, D, o = env
    say(f"lm_head M={M} d={d} V={V}")
    t = _table(V, d, key=(41, d, V))
    E, scale = table_1p3b if t is None else t
    x = S.activations(M, d, key=(42, M, d))
    q, s = o.quantize_act(x)
    _check_lm(torch, D, o, q, s, E, scale, f"M={M} d={d} V={V}")


@pytest.mark.parametrize("M,d,V,threshold", [(1, 2048, 1001, 1), (3, 256, 77, 1), (64, 2048, 1001, 100000),
                                              (20, 768, 333, 100000)])
def test_lm_head_both_kernels(env, M, d, V, threshold):
    # the test switch moves the token count from which the matrix-core
    # kernel runs: few tokens through it, many through the GEMV passes
    torch, D, o = env
    say(f"lm_head M={M} d={d} V={V} threshold={threshold}")
    E, scale = S.embedding(V, d, key=(49, d, V))
    q, s = o.quantize_act(S.activations(M, d, key=(49, M, d)))
    with forced_switch(D, D.TEST_LM_HEAD_MFMA_TOKENS, threshold):
        _check_lm(torch, D, o, q, s, E, scale, f"M={M} d={d} V={V} threshold={threshold}")


@pytest.mark.parametrize("M,d,V,threshold", [(8, 2048, 1001, 8), (17, 1024, 77, 8), (64, 2048, 1001, 100000),
                                              (300, 768, 1001, 100000)])
def test_lm_head_tiled_switch(env, M, d, V, threshold):
    # the test switch moves the token count from which the matrix-core path
    # runs the tiled kernel: few tokens through it, many through the kernel
    # that holds the table slice in registers
    torch, D, o = env
    say(f"lm_head tiled switch M={M} d={d} V={V} threshold={threshold}")
    E, scale = S.embedding(V, d, key=(50, d, V))
    q, s = o.quantize_act(S.activations(M, d, key=(50, M, d)))
    with forced_switch(D, D.TEST_LM_HEAD_TILED_TOKENS, threshold):
        _check_lm(torch, D, o, q, s, E, scale, f"M={M} d={d} V={V} tiled threshold={threshold}")


def test_lm_head_extremes(env):
    # |acc| at its largest (127 * 127 * 16384 = 264,257,536) and values past
    # 2^24, where (float)acc rounds: int32 exactness and the rounding order
    torch, D, o = env
    say("lm_head extremes")
    d, V = 16384, 8
    E = np.full((V, d), 127, np.int8)
    E[1] = -127
    E[2, ::2] = -127
    E[3] = np.tile(np.array([127, -127, 1, 0], np.int8), d // 4)
    g = np.random.default_rng(43)
    E[4:] = g.integers(-127, 128, size=(V - 4, d), dtype=np.int8)
    scale = np.array([1.0, 3.0, 0.1, 7e-4, 1e-20, 2.5e29, 1.0, 0.3], np.float32)
    q = np.full((3, d), 127, np.int8)
    q[1] = -127
    q[2] = g.integers(-127, 128, size=d, dtype=np.int8)
    s = np.array([1.0 / 127, 0.37, 0.0], np.float32)
    _check_lm(torch, D, o, q, s, E, scale, "extremes")


def test_lm_head_outputs_optional(env):
    torch, D, o = env
    say("lm_head optional outputs")
    M, d, V = 2, 256, 77
    E, scale = S.embedding(V, d, key=(44,))
    q, s = o.quantize_act(S.activations(M, d, key=(44,)))
    acc_r, lg_r = o.lm_head(q, s, E, scale)
    qd, sd, Ed, scd = dev(q), dev(s), dev(E), dev(scale)
    lg = torch.full((M, V), 7.0, dtype=torch.float32, device="cuda")
    acc = torch.full((M, V), 7, dtype=torch.int32, device="cuda")
    D._check(D.lib.dfssm_lm_head(qd.data_ptr(), sd.data_ptr(), M, d, Ed.data_ptr(), scd.data_ptr(), V,
                                 lg.data_ptr(), None, None))
    D._check(D.lib.dfssm_lm_head(qd.data_ptr(), sd.data_ptr(), M, d, Ed.data_ptr(), scd.data_ptr(), V,
                                 None, acc.data_ptr(), None))
    torch.cuda.synchronize()
    assert np.array_equal(host(acc), acc_r)
    assert np.array_equal(host(lg).view(np.uint32), lg_r.view(np.uint32))
    # empty problems write nothing
    D._check(D.lib.dfssm_lm_head(qd.data_ptr(), sd.data_ptr(), 0, d, Ed.data_ptr(), scd.data_ptr(), V,
                                 lg.data_ptr(), None, None))
    D._check(D.lib.dfssm_lm_head(qd.data_ptr(), sd.data_ptr(), M, d, Ed.data_ptr(), scd.data_ptr(), 0,
                                 lg.data_ptr(), None, None))
    torch.cuda.synchronize()
    assert np.array_equal(host(lg).view(np.uint32), lg_r.view(np.uint32))


def test_lm_head_end_to_end(env, table_1p3b):
    # final hidden state -> per-token quantiser -> LM head, all on the device
    torch, D, o = env
    say("lm_head end to end")
    E, scale = table_1p3b
    x = S.activations(2, S.D_MODEL_1P3B, key=(45,))
    q, s = o.quantize_act(x)
    acc_r, lg_r = o.lm_head(q, s, E, scale)
    qd, sd = D.quantize_act(dev(x))
    lg = D.lm_head(qd, sd, dev(E), dev(scale))
    torch.cuda.synchronize()
    assert np.array_equal(host(lg).view(np.uint32), lg_r.view(np.uint32))
    assert np.array_equal(np.argmax(host(lg), axis=1), np.argmax(lg_r, axis=1))


# ---------------------------------------------------------------- gather
GSHAPES = [
    # (V, d, M)
    (50280, 2048, 4),
    (50280, 2048, 1),
    (1000, 768, 37),
    (37, 16, 3),
    (100, 2064, 7),
    (64, 65536, 2),     # the longest row
]


@pytest.mark.parametrize("V,d,M", GSHAPES)
def test_embed_gather(env, table_1p3b, V, d, M):
    torch, D, o = env
    say(f"embed_gather V={V} d={d} M={M}")
    t = _table(V, d, key=(46, V, d))
    E, scale = table_1p3b if t is None else t
    tok = S.tokens(M, V, key=(47, V, M))
    xr = o.embed_gather(E, scale, tok)
    x = D.embed_gather(dev(E), dev(scale), dev(tok))
    torch.cuda.synchronize()
    assert np.array_equal(host(x).view(np.uint32), xr.view(np.uint32))


def test_embed_gather_ids_outside_table(env):
    torch, D, o = env
    say("embed_gather ids outside the table")
    V, d = 50, 64
    E, scale = S.embedding(V, d, key=(48,))
    tok = np.array([3, -1, V, 0, V - 1, 2 ** 31 - 1, -2 ** 31, 7], np.int32)
    ok = (tok >= 0) & (tok < V)
    xr = o.embed_gather(E, scale, tok[ok])
    x = host(D.embed_gather(dev(E), dev(scale), dev(tok)))
    torch.cuda.synchronize()
    assert np.array_equal(x[ok].view(np.uint32), xr.view(np.uint32))
    assert np.all(x[~ok].view(np.uint32) == 0)
