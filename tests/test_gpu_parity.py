"""GPU parity: the HIP library (through its C ABI) against the CPU oracle on
the same seeded inputs.  Integers (Q, acc_s, acc_a, acc_b) must match
bit-exactly; y must be within 1e-3 * max|y| of the fp64 oracle and is also
checked bit-exact against the oracle's fp32 evaluation in the same order."""
import numpy as np
import pytest

import dfssm_synth as S
import oracle
from gpu_util import assert_y, dev, dev_weights, forced_switch, host, say, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch = torch_cuda()
    import paper_2606_10932_amd as D
    oracle.build()
    return torch, D, oracle.get()


# ---------------------------------------------------------------- quantiser
QSHAPES = [(1, 768, 768), (1, 2048, 2048), (3, 4096, 4096), (5, 32, 32), (2, 96, 96),
           (4, 64, 72), (2, 128, 131), (64, 2048, 2048)]


@pytest.mark.parametrize("dtype", ["f16", "f32"])
@pytest.mark.parametrize("M,K,ldx", QSHAPES)
def test_quantize(env, dtype, M, K, ldx):
    torch, D, o = env
    say(f"quantize {dtype} M={M} K={K} ldx={ldx}")
    x = S.activations(M, ldx, key=(10, M, K, ldx))
    x = x if dtype == "f16" else (x.astype(np.float32) * np.float32(3.7))
    if M > 2:
        x[1, :] = 0  # an all-zero row
    qr, sr = o.quantize_act(x, K=K)
    xd = dev(x)
    q, s = D.quantize_act(xd[:, :K] if ldx != K else xd, K=K)
    torch.cuda.synchronize()
    assert np.array_equal(host(q), qr)
    assert np.array_equal(host(s).view(np.uint32), sr.view(np.uint32))


def test_quantize_ties_and_subnormals(env):
    torch, D, o = env
    say("quantize ties/subnormals")
    x = np.zeros((3, 32), np.float32)
    x[0, :8] = [0.5, 1.5, 2.5, -0.5, -2.5, 126.5, -126.5, 127.0]
    x[1, :2] = [1.375, 0.6875]
    x[2, 3] = 1e-40
    qr, sr = o.quantize_act(x)
    q, s = D.quantize_act(dev(x))
    torch.cuda.synchronize()
    assert np.array_equal(host(q), qr) and np.array_equal(host(s), sr)


# ---------------------------------------------------------------- the linear
LSHAPES = [
    # (M, K, N, r)  -- several tiles, ragged tails, both families
    (1, 768, 3352, 16),      # Mamba-2-130M in_proj
    (1, 2048, 8512, 64),     # Mamba-2-1.3B in_proj
    (1, 4096, 2048, 64),     # Mamba-2-1.3B out_proj
    (2, 4096, 2048, 64),
    (3, 2048, 333, 64),
    (4, 4096, 2048, 64),
    (5, 160, 77, 5),         # K % 128 != 0, r % 4 != 0
    (1, 32, 1, 0),
    (3, 96, 33, 1),
    (2, 256, 31, 256),
    (7, 8192, 130, 64),
    (1, 12288, 70, 32),      # two chunks per lane
    (2, 20480, 40, 8),       # planes streamed from memory
    (33, 128, 130, 64),
    (130, 2048, 300, 64),
    (16, 4096, 2048, 64),
]


def _run_linear(env, M, K, N, r, path, beta_scale=1.0, key=0):
    torch, D, o = env
    ws = S.weights(K, N, r, key=(11, M, K, N, r, key), beta_scale=beta_scale)
    x = S.activations(M, K, key=(11, M, K, key))
    q, s = o.quantize_act(x)
    ref = o.linear(q, s, **ws)
    d = dev_weights(ws)
    y, acc_s, acc_a, acc_b = D.scaffold_lora_linear(dev(q), dev(s), d["w_bits"], d["alpha"], d["A"], d["B"],
                                                    d["beta"], path=path, acc=True)
    torch.cuda.synchronize()
    return ref, host(y), host(acc_s), host(acc_a), host(acc_b)


def _run_y_only(env, M, K, N, r, path, key=0):
    torch, D, o = env
    ws = S.weights(K, N, r, key=(11, M, K, N, r, key))
    q, s = o.quantize_act(S.activations(M, K, key=(11, M, K, key)))
    d = dev_weights(ws)
    y = D.scaffold_lora_linear(dev(q), dev(s), d["w_bits"], d["alpha"], d["A"], d["B"], d["beta"], path=path)
    torch.cuda.synchronize()
    return host(y)


@pytest.mark.parametrize("path", ["decode", "mfma"])
@pytest.mark.parametrize("M,K,N,r", LSHAPES)
def test_linear(env, path, M, K, N, r):
    torch, D, o = env
    say(f"linear path={path} M={M} K={K} N={N} r={r}")
    p = D.PATH_DECODE if path == "decode" else D.PATH_MFMA
    ref, y, acc_s, acc_a, acc_b = _run_linear(env, M, K, N, r, p)
    assert np.array_equal(acc_s, ref["acc_s"]), "acc_s"
    if r:
        assert np.array_equal(acc_a, ref["acc_a"]), "acc_a"
    assert np.array_equal(acc_b, ref["acc_b"]), "acc_b"
    assert_y(y, ref, what=f"{path} {M}x{K}x{N} r{r}")
    # without accumulator outputs the kernels take their unchecked epilogue
    # on whole tiles: the same y, bit for bit
    y2 = _run_y_only(env, M, K, N, r, p)
    assert np.array_equal(y2.view(np.uint32), y.view(np.uint32)), "y without accumulator outputs"


def _with_int8_min(ws: dict, key) -> dict:
    """-128 planted in A and B (int8 storage admits it; the seeded draw stops
    at -127): a whole row of A, every 7th column of A, a whole row of B and
    every 5th row of B in one rank."""
    w = {k: v.copy() for k, v in ws.items()}
    A, B = w["A"], w["B"]
    g = np.random.default_rng(list(key))
    A[g.integers(A.shape[0])] = -128
    A[:, ::7] = -128
    B[g.integers(B.shape[0])] = -128
    B[::5, g.integers(B.shape[1])] = -128
    return w


@pytest.mark.parametrize("path", ["few", "decode", "mfma4", "mfma8"])
@pytest.mark.parametrize("M,K,N,r", [(1, 2048, 8512, 64), (3, 4096, 2048, 64), (70, 2048, 300, 64),
                                     (130, 4096, 2048, 256), (5, 160, 77, 5)])
def test_linear_int8_min(env, path, M, K, N, r):
    """-128 in the LoRA factors on every kernel family: the exact integers
    and y against the oracle (A at -128 everywhere in a row drives acc_a to
    its extreme for that rank)."""
    torch, D, o = env
    if path == "few" and M > 512:
        pytest.skip("few-token path takes M <= 512")
    say(f"linear int8 min path={path} M={M} K={K} N={N} r={r}")
    ws = _with_int8_min(S.weights(K, N, r, key=(12, M, K, N, r)), (12, M, K))
    assert (ws["A"] == -128).any() and (ws["B"] == -128).any()
    q, s = o.quantize_act(S.activations(M, K, key=(12, M, K)))
    ref = o.linear(q, s, **ws)
    d = dev_weights(ws)
    p = {"few": D.PATH_MFMA_FEW, "decode": D.PATH_DECODE}.get(path, D.PATH_MFMA)
    forced = {"mfma4": 4, "mfma8": 8}.get(path, 0)
    with forced_switch(D, D.TEST_PREFILL_KERNEL, forced):
        y, acc_s, acc_a, acc_b = D.scaffold_lora_linear(dev(q), dev(s), d["w_bits"], d["alpha"], d["A"], d["B"],
                                                        d["beta"], path=p, acc=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(acc_s), ref["acc_s"]), "acc_s"
    assert np.array_equal(host(acc_a), ref["acc_a"]), "acc_a"
    assert np.array_equal(host(acc_b), ref["acc_b"]), "acc_b"
    assert_y(host(y), ref, what=f"int8 min {path} {M}x{K}x{N} r{r}")


# few-token MFMA path (M <= 512; up to 32 tokens 1 or 2 token tiles per
# workgroup, above 32 blocks of 64 tokens, 4 tiles): 8- and 16-byte sign loads, K splits of one or more iterations per
# wave, unaligned sign rows, ragged N, rank 0, rank not a multiple of 16 and
# ranks above 64, several chunks with a ragged last one
FSHAPES = [
    (1, 768, 3352, 16),      # Mamba-2-130M in_proj: 3 waves
    (1, 2048, 8512, 64),     # Mamba-2-1.3B in_proj
    (4, 2048, 8512, 64),     # the most tokens the copies' token-major polls take (int8)
    (5, 4096, 2048, 64),     # Mamba-2-1.3B out_proj, small batches
    (7, 2048, 8512, 64),     # the copies polled by two waves together, the second with 3 tokens
    (8, 2048, 8512, 64),
    (13, 2048, 8512, 64),    # above 8 tokens: one copy again
    (16, 4096, 2048, 64),
    (17, 4096, 2048, 64),
    (32, 4096, 2048, 64),
    (3, 160, 77, 5),         # odd sign-row length, N % 4 != 0, r % 16 != 0
    (1, 32, 1, 0),
    (9, 96, 33, 1),
    (2, 256, 31, 256),       # four 64-rank chunks
    (20, 8192, 130, 64),     # two iterations per wave
    (32, 4128, 50, 72),      # K % 512 != 0 with 16-byte sign loads, odd row length
    (12, 12288, 70, 32),
    (31, 2048, 300, 64),
    (33, 2048, 8512, 64),    # one 64-token block holding 33 tokens
    (65, 4096, 2048, 64),    # two blocks, the second of one token
    (96, 4096, 2048, 64),    # two blocks, the second of two full tiles
    (100, 160, 77, 5),       # ragged last block, odd shapes
    (130, 4096, 2048, 64),   # three blocks, out_proj shape
    (200, 256, 31, 256),
    (512, 96, 33, 1),        # the largest M the path takes
]


@pytest.mark.parametrize("M,K,N,r", FSHAPES)
def test_linear_few_tokens(env, M, K, N, r):
    torch, D, o = env
    say(f"linear path=few M={M} K={K} N={N} r={r}")
    ref, y, acc_s, acc_a, acc_b = _run_linear(env, M, K, N, r, D.PATH_MFMA_FEW)
    assert np.array_equal(acc_s, ref["acc_s"]), "acc_s"
    if r:
        assert np.array_equal(acc_a, ref["acc_a"]), "acc_a"
    assert np.array_equal(acc_b, ref["acc_b"]), "acc_b"
    assert_y(y, ref, what=f"few {M}x{K}x{N} r{r}")
    y2 = _run_y_only(env, M, K, N, r, D.PATH_MFMA_FEW)
    assert np.array_equal(y2.view(np.uint32), y.view(np.uint32)), "y without accumulator outputs"


@pytest.mark.parametrize("M,K,N,r", [(3, 160, 77, 5), (17, 4096, 2048, 64), (2, 256, 31, 256), (1, 32, 1, 0),
                                     (70, 2048, 300, 64)])
def test_few_tokens_local_lora(env, M, K, N, r):
    """The few-token kernel's fallback: with no LoRA workgroups launched and
    no polling (a test switch of the library), every lane computes acc_a and
    sum Q itself; the results are the same integers."""
    torch, D, o = env
    say(f"few tokens, local LoRA values M={M} K={K} N={N} r={r}")
    with forced_switch(D, D.TEST_LOCAL_LORA, 1):
        ref, y, acc_s, acc_a, acc_b = _run_linear(env, M, K, N, r, D.PATH_MFMA_FEW)
    assert np.array_equal(acc_s, ref["acc_s"]), "acc_s"
    if r:
        assert np.array_equal(acc_a, ref["acc_a"]), "acc_a"
    assert np.array_equal(acc_b, ref["acc_b"]), "acc_b"
    assert_y(y, ref, what=f"few local {M}x{K}x{N} r{r}")


def test_few_tokens_limit(env):
    """The few-token path refuses M > 512 before launching anything."""
    torch, D, o = env
    ws = dev_weights(S.weights(64, 16, 4, key=(14,)))
    q = torch.zeros((513, 64), dtype=torch.int8, device="cuda")
    s = torch.zeros((513,), dtype=torch.float32, device="cuda")
    with pytest.raises(D.DfssmError):
        D.scaffold_lora_linear(q, s, ws["w_bits"], ws["alpha"], ws["A"], ws["B"], ws["beta"], path=D.PATH_MFMA_FEW)


@pytest.mark.parametrize("M", [1, 4, 8, 16, 32])
def test_out_proj_small_batch_auto(env, M):
    """Mamba-2-1.3B out_proj at the small-batch decode sizes, automatic path."""
    say(f"out_proj auto M={M}")
    ref, y, acc_s, acc_a, acc_b = _run_linear(env, M, 4096, 2048, 64, 0, key=M)
    assert np.array_equal(acc_s, ref["acc_s"]) and np.array_equal(acc_b, ref["acc_b"])
    assert_y(y, ref, what=f"out_proj M={M}")


@pytest.mark.parametrize("path", ["decode", "mfma"])
def test_realistic_lora_ratio(env, path):
    """beta scaled so the LoRA term is ~1.5% of the scaffold term (the trained
    model's ratio) -- y then depends visibly on the scaffold product."""
    torch, D, o = env
    say(f"realistic ratio {path}")
    p = D.PATH_DECODE if path == "decode" else D.PATH_MFMA
    ref, y, acc_s, _, acc_b = _run_linear(env, 2, 2048, 8512, 64, p, beta_scale=1.8e-5)
    assert np.array_equal(acc_s, ref["acc_s"]) and np.array_equal(acc_b, ref["acc_b"])
    assert_y(y, ref, what="realistic ratio")


# the two prefill kernels (4-wave blocks, two per CU; 8-wave ping-pong
# blocks, one per CU) on shapes the automatic choice would not give them
PSHAPES = [
    (5, 160, 77, 5),         # K % 128 != 0, r % 4 != 0
    (33, 128, 130, 64),
    (130, 2048, 300, 64),
    (16, 4096, 2048, 64),
    (2, 256, 31, 256),       # ranks above 64: LoRA operands from memory
    (300, 2080, 700, 64),    # K % 64 == 32: half last stage
    (129, 96, 600, 0),       # no LoRA, 2-stage K
    # 9 slices: runs of 4-5 row tiles take the 8-row short form, runs of 8-9
    # the full form (smaller shapes take the 4-row short form)
    (1100, 288, 4201, 64),   # short, 8-row form; K % 64 == 32, ragged N
    (1030, 256, 4200, 0),
    (1100, 288, 7400, 64),   # full form
    (1030, 256, 7300, 0),
]


@pytest.mark.parametrize("kernel", ["4", "8"])
@pytest.mark.parametrize("M,K,N,r", PSHAPES)
def test_linear_prefill_kernels(env, kernel, M, K, N, r):
    torch, D, o = env
    say(f"prefill kernel={kernel} M={M} K={K} N={N} r={r}")
    with forced_switch(D, D.TEST_PREFILL_KERNEL, int(kernel)):
        ref, y, acc_s, acc_a, acc_b = _run_linear(env, M, K, N, r, D.PATH_MFMA)
        y2 = _run_y_only(env, M, K, N, r, D.PATH_MFMA)
    assert np.array_equal(acc_s, ref["acc_s"]), "acc_s"
    if r:
        assert np.array_equal(acc_a, ref["acc_a"]), "acc_a"
    assert np.array_equal(acc_b, ref["acc_b"]), "acc_b"
    assert_y(y, ref, what=f"prefill{kernel} {M}x{K}x{N} r{r}")
    assert np.array_equal(y2.view(np.uint32), y.view(np.uint32)), "y without accumulator outputs"


# the 4-wave kernel's short forms (every run of the grid at most 4, or at
# most 8, row tiles: wave w multiplies token tiles 2w, 2w+1 of each row
# tile and skips tiles past M), as the prefill path takes them at a few
# hundred tokens
SHORT_SHAPES = [
    (100, 2048, 8512, 64),   # 1.3B in_proj, one partial 128-token slice
    (33, 768, 3352, 16),     # 130M in_proj, 3 token tiles
    (500, 1536, 768, 64),    # 130M out_proj, 4 slices, the last partial
    (200, 4096, 2048, 72),   # ranks above 64: LoRA operands from memory
    (77, 2080, 210, 0),      # no LoRA, K % 64 == 32, ragged N
    (260, 4096, 2048, 64),   # 1.3B out_proj, 3 slices
    (300, 256, 10900, 64),   # runs of 3-4 row tiles, ragged N
    (512, 2048, 8512, 64),   # 1.3B in_proj, runs of 4-5: the 8-row form
    (1100, 256, 4200, 72),   # the 8-row form, ranks above 64
]


@pytest.mark.parametrize("M,K,N,r", SHORT_SHAPES)
def test_linear_prefill_short_form(env, M, K, N, r):
    torch, D, o = env
    say(f"prefill short form M={M} K={K} N={N} r={r}")
    with forced_switch(D, D.TEST_PREFILL_KERNEL, 4):
        ref, y, acc_s, acc_a, acc_b = _run_linear(env, M, K, N, r, D.PATH_MFMA)
        y2 = _run_y_only(env, M, K, N, r, D.PATH_MFMA)
    assert np.array_equal(acc_s, ref["acc_s"]), "acc_s"
    if r:
        assert np.array_equal(acc_a, ref["acc_a"]), "acc_a"
    assert np.array_equal(acc_b, ref["acc_b"]), "acc_b"
    assert_y(y, ref, what=f"short {M}x{K}x{N} r{r}")
    assert np.array_equal(y2.view(np.uint32), y.view(np.uint32)), "y without accumulator outputs"
    # the automatic path at this size (few-token or prefill, by the cost model)
    ya = _run_y_only(env, M, K, N, r, D.PATH_AUTO)
    assert np.array_equal(ya.view(np.uint32), y.view(np.uint32)), "automatic path"


@pytest.mark.parametrize("kernel", [0, 4])
def test_prefill_full_size(env, kernel):
    """Mamba-2-1.3B in_proj at 2048 tokens (the launch the benchmark times,
    which takes the 8-wave kernel; and the 4-wave kernel on the same shape):
    every acc_s/acc_a/acc_b and y of all 2048 token rows against the oracle."""
    torch, D, o = env
    M, K, N, r = 2048, 2048, 8512, 64
    say(f"prefill {M}x{K}x{N} r{r} kernel={kernel or 'auto'}")
    ws = S.config_weights(4)
    x = S.config_activations(4, M)
    q, s = o.quantize_act(x)
    d = dev_weights(ws)
    qd, sd = D.quantize_act(dev(x))
    with forced_switch(D, D.TEST_PREFILL_KERNEL, kernel):
        y, acc_s, acc_a, acc_b = D.scaffold_lora_linear(qd, sd, d["w_bits"], d["alpha"], d["A"], d["B"], d["beta"],
                                                        acc=True)
        # the benchmark's call (no accumulator outputs: unchecked epilogue on
        # whole tiles)
        y2 = D.scaffold_lora_linear(qd, sd, d["w_bits"], d["alpha"], d["A"], d["B"], d["beta"])
    torch.cuda.synchronize()
    assert np.array_equal(host(qd), q) and np.array_equal(host(sd), s)
    ref = o.linear(q, s, **ws)
    for name, got in (("acc_s", acc_s), ("acc_a", acc_a), ("acc_b", acc_b)):
        bad = np.argwhere(host(got) != ref[name])
        assert bad.size == 0, f"{name}: {len(bad)} entries differ, first {bad[:4].tolist()}"
    assert_y(host(y), ref, what="prefill 2048 tokens")
    assert torch.equal(y, y2)


@pytest.mark.parametrize("K", [2080, 2048])
def test_prefill_ragged_sampled(env, K):
    """A prefill-sized linear with ragged tails: tokens past a whole 128-row
    tile and output rows past a whole 16-row tile; K = 2080 adds a 32-column
    last stage (general kernel), K = 2048 takes the wide kernel with its
    shared 33rd and 34th row tiles.  Sampled rows (including the partial
    token tile) against the oracle; the y of the call without accumulator
    outputs equals the checked one everywhere."""
    torch, D, o = env
    M, N, r = 2085, 8532, 64
    say(f"prefill ragged {M}x{K}x{N} r{r}")
    ws = S.weights(K, N, r, key=(13, K))
    x = S.activations(M, K, key=(13, K))
    q, s = o.quantize_act(x)
    d = dev_weights(ws)
    qd, sd = dev(q), dev(s)
    y, acc_s, acc_a, acc_b = D.scaffold_lora_linear(qd, sd, d["w_bits"], d["alpha"], d["A"], d["B"], d["beta"],
                                                    acc=True)
    y2 = D.scaffold_lora_linear(qd, sd, d["w_bits"], d["alpha"], d["A"], d["B"], d["beta"])
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 127, 128, 2047, 2048, 2060, M - 1],
                                     np.random.default_rng(1).choice(M, 17, replace=False)]))
    ref = o.linear(q[rows], s[rows], **ws)
    assert np.array_equal(host(acc_s)[rows], ref["acc_s"])
    assert np.array_equal(host(acc_a)[rows], ref["acc_a"])
    assert np.array_equal(host(acc_b)[rows], ref["acc_b"])
    assert_y(host(y)[rows], ref, what="ragged prefill sample")
    assert torch.equal(y, y2)


def test_edge_cases(env):
    torch, D, o = env
    say("edge cases")
    K, N, r = 256, 40, 8
    ws = S.weights(K, N, r, key=(12,))
    d = dev_weights(ws)
    # M = 0 and N = 0 are no-ops
    q0 = torch.empty((0, K), dtype=torch.int8, device="cuda")
    s0 = torch.empty((0,), dtype=torch.float32, device="cuda")
    y = D.scaffold_lora_linear(q0, s0, d["w_bits"], d["alpha"], d["A"], d["B"], d["beta"])
    assert y.shape == (0, N)
    # all-zero activations -> y = 0; A = 0 -> scaffold only
    for path in (D.PATH_DECODE, D.PATH_MFMA, D.PATH_MFMA_FEW):
        x = np.zeros((3, K), np.float32)
        x[1] = S.activations(1, K, key=(12, 1))[0]
        q, s = o.quantize_act(x)
        Az = np.zeros_like(ws["A"])
        ref = o.linear(q, s, ws["w_bits"], ws["alpha"], Az, ws["B"], ws["beta"])
        y, acc_s, acc_a, acc_b = D.scaffold_lora_linear(dev(q), dev(s), d["w_bits"], d["alpha"], dev(Az),
                                                        d["B"], d["beta"], path=path, acc=True)
        torch.cuda.synchronize()
        assert not host(y)[0].any() and not host(y)[2].any()
        assert np.array_equal(host(acc_s), ref["acc_s"]) and not host(acc_b).any()
        assert_y(host(y), ref, what="A=0")


def test_deterministic_and_streams(env):
    """Bitwise identical repeats, on the default stream and on a side stream
    ordered by events."""
    torch, D, o = env
    say("determinism")
    ws = S.config_weights(1)
    d = dev_weights(ws)
    q, s = D.quantize_act(dev(S.config_activations(1, 1)))
    y1 = D.scaffold_lora_linear(q, s, d["w_bits"], d["alpha"], d["A"], d["B"], d["beta"])
    side = torch.cuda.Stream()
    ev = torch.cuda.Event()
    ev.record()
    with torch.cuda.stream(side):
        side.wait_event(ev)
        y2 = D.scaffold_lora_linear(q, s, d["w_bits"], d["alpha"], d["A"], d["B"], d["beta"])
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
