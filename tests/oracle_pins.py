"""Pins for the CPU oracle: checks against facts that do not come from the
oracle itself (hand-derived cases, closed forms, invariants, brute force with
an independent unpack route, the paper's printed sizes).

Each pin takes an ``oracle.Oracle`` and raises AssertionError on a mismatch.
They are written as plain functions so the same set can be run against the
real oracle and against deliberately broken copies of it (planted mistakes),
proving that a plausible mistake anywhere in the oracle fails at least one.
"""
from __future__ import annotations

import json
import os

import numpy as np

import dfssm_synth as S
from oracle import Oracle, OracleError, ERR_NONFINITE

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
F32 = np.float32


# --------------------------------------------------------------------------
# independent helpers (no oracle code): unpack through numpy's bit routines
# --------------------------------------------------------------------------
def unpack_signs(w_bits: np.ndarray) -> np.ndarray:
    """[N, K/32] uint32 -> [N, K] int64 +-1, via numpy.unpackbits on the
    little-endian byte view (bit j of word w is column 32w + j)."""
    N, W = w_bits.shape
    b = np.unpackbits(w_bits.astype("<u4").view(np.uint8).reshape(N, W * 4), axis=1, bitorder="little")
    return b.astype(np.int64) * 2 - 1


def pack_signs(S_pm1: np.ndarray) -> np.ndarray:
    """[N, K] +-1 -> [N, K/32] uint32 (inverse of unpack_signs)."""
    N, K = S_pm1.shape
    b = (S_pm1 > 0).astype(np.uint8)
    by = np.ascontiguousarray(np.packbits(b, axis=1, bitorder="little"))
    return by.view("<u4").reshape(N, K // 32).astype(np.uint32)


def bruteforce_int(q, w_bits, A, B):
    Sd = unpack_signs(w_bits)
    q64 = q.astype(np.int64)
    acc_s = q64 @ Sd.T
    acc_a = q64 @ A.astype(np.int64).T if A is not None and A.shape[0] else np.zeros((q.shape[0], 0), np.int64)
    acc_b = acc_a @ B.astype(np.int64).T if A is not None and A.shape[0] else np.zeros_like(acc_s)
    return acc_s, acc_a, acc_b


def _case(M, K, N, r, seed, beta_scale=1.0):
    ws = S.weights(K, N, r, key=(90, seed, K, N), beta_scale=beta_scale)
    x = S.activations(M, K, key=(90, seed))
    return ws, x


# --------------------------------------------------------------------------
# fp16 decode
# --------------------------------------------------------------------------
def pin_f16_decode(o: Oracle):
    """Every binary16 pattern decodes to numpy's (IEEE) float16 -> float32."""
    pats = np.arange(65536, dtype=np.uint16)
    ref = pats.view(np.float16).astype(np.float32)
    got = np.array([o.f16_to_f32(int(p)) for p in pats[::1]], np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan), "NaN patterns"
    assert np.array_equal(got[~nan].view(np.uint32), ref[~nan].view(np.uint32)), "binary16 decode"


# --------------------------------------------------------------------------
# quantiser
# --------------------------------------------------------------------------
def pin_quantize_hand_cases(o: Oracle):
    """Hand-derived cases (absmax a, inv = 127/a, Q = rint(x*inv))."""
    # a = 4, inv = 31.75 exactly; 1*31.75 = 31.75 -> 32; -2*31.75 = -63.5 ->
    # -64 (tie, even); 0.5*31.75 = 15.875 -> 16; 4*31.75 = 127.
    x = np.zeros((1, 32), F32)
    x[0, :4] = [1.0, -2.0, 0.5, 4.0]
    q, s = o.quantize_act(x)
    assert q[0, :4].tolist() == [32, -64, 16, 127] and not q[0, 4:].any()
    assert s[0] == F32(4.0) / F32(127.0)
    # a = 127, inv = 1: Q = rint(x), ties to even: 0.5->0, 1.5->2, 2.5->2,
    # -0.5->-0, -2.5->-2, 126.5->126, -126.5 -> -126
    x = np.zeros((1, 32), F32)
    x[0, :8] = [0.5, 1.5, 2.5, -0.5, -2.5, 126.5, -126.5, 127.0]
    q, s = o.quantize_act(x)
    assert q[0, :8].tolist() == [0, 2, 2, 0, -2, 126, -126, 127]
    assert s[0] == F32(1.0)
    # a = 254, inv = 0.5: 3 -> 1.5 -> 2; 5 -> 2.5 -> 2; -7 -> -3.5 -> -4;
    # -254 -> -127; s = 2
    x = np.zeros((1, 32), F32)
    x[0, :4] = [3.0, 5.0, -7.0, -254.0]
    q, s = o.quantize_act(x)
    assert q[0, :4].tolist() == [2, 2, -4, -127] and s[0] == F32(2.0)
    # two rows, fp16 input, row stride 40 > K = 32 (stride must be honoured)
    x = np.zeros((2, 40), np.float16)
    x[0, :2] = [2.0, -1.0]
    x[0, 32:] = 1000.0          # beyond K: must not enter the absmax
    x[1, 31] = -0.25
    q, s = o.quantize_act(x, K=32)
    assert q[0, :2].tolist() == [127, -64] and s[0] == F32(2.0) / F32(127.0)  # -63.5 -> -64
    assert q[1, 31] == -127 and not q[1, :31].any() and s[1] == F32(0.25) / F32(127.0)
    # the multiplier is the fp32 quotient 127/a, not 1/s: a = 1.375 = 11/8,
    # 127/a = 1016/11 = 92.3636...; its fp32 neighbours are 6053143/65536
    # (4.2e-6 below) and 12106287/131072 (3.5e-6 above), so inv rounds up to
    # 12106287/131072.  x = 0.6875 = a/2: x*inv = 133169157/2097152 =
    # 63.5000024 (exact product, fits fp32) -> rint 64.  Dividing by
    # s = fp32(a/127) instead gives 63.499996 -> 63.
    x = np.zeros((1, 32), F32)
    x[0, :2] = [1.375, 0.6875]
    q, s = o.quantize_act(x)
    assert q[0, :2].tolist() == [127, 64]


def pin_quantize_properties(o: Oracle):
    g = np.random.default_rng(7)
    for trial in range(20):
        K = 32 * int(g.integers(1, 9))
        x = (g.standard_normal((3, K)) * 10.0 ** g.uniform(-3, 3)).astype(F32)
        q, s = o.quantize_act(x)
        assert np.abs(q.astype(int)).max() <= 127
        for m in range(3):
            a = np.abs(x[m]).max()
            i = int(np.argmax(np.abs(x[m])))
            assert abs(int(q[m, i])) == 127 and np.sign(q[m, i]) == np.sign(x[m, i]), "argmax -> +-127"
            # reconstruction error of a round-to-nearest quantiser: |x - s*Q| <= s/2 (+ fp32 slack)
            err = np.abs(x[m].astype(np.float64) - float(s[m]) * q[m].astype(np.float64))
            assert err.max() <= 0.5 * float(s[m]) * (1 + 1e-4), "reconstruction bound"
            assert s[m] == F32(a) / F32(127.0)
            # monotone and odd
            order = np.argsort(x[m], kind="stable")
            assert np.all(np.diff(q[m, order].astype(int)) >= 0), "monotone"
        qn, sn = o.quantize_act(-x)
        assert np.array_equal(qn, -q) and np.array_equal(sn, s), "odd symmetry"
        # scaling by 2^e changes nothing but s (exactly)
        e = int(g.integers(-8, 9))
        q2, s2 = o.quantize_act((x * F32(2.0 ** e)).astype(F32))
        assert np.array_equal(q2, q) and np.array_equal(s2, s * F32(2.0 ** e)), "2^e invariance"
    # zero and subnormal rows -> Q = 0, s = 0
    x = np.zeros((2, 64), F32)
    x[1, 5] = 1e-40
    q, s = o.quantize_act(x)
    assert not q.any() and not s.any()
    # fp16 and fp32 input holding the same values agree
    xh = S.activations(4, 96, key=(91, 0))
    qa, sa = o.quantize_act(xh)
    qb, sb = o.quantize_act(xh.astype(F32))
    assert np.array_equal(qa, qb) and np.array_equal(sa, sb)
    # non-finite input is refused
    for bad in (np.inf, -np.inf, np.nan):
        x = np.ones((1, 32), F32)
        x[0, 3] = bad
        try:
            o.quantize_act(x)
        except OracleError as e:
            assert e.status == ERR_NONFINITE
        else:
            raise AssertionError("non-finite accepted")


# --------------------------------------------------------------------------
# the linear: integer accumulators
# --------------------------------------------------------------------------
def pin_hand_linear(o: Oracle):
    """K = 32, N = 2, r = 1, M = 1, worked by hand.
    Q = [1, 2, ..., 32]; sum Q = 528.
    row 0: word 0x0000000F -> columns 0..3 are +1: 2*(1+2+3+4) - 528 = -508
    row 1: word 0x80000001 -> columns 0 and 31: 2*(1+32) - 528 = -462
    A = [1, -1, 1, -1, ...] -> acc_a = sum_k (-1)^k (k+1) = -16
    B = [[3], [-2]] -> acc_b = [-48, 32]
    alpha = [0.5, 0.25], beta = [0.125, 1.0], s = 2:
      y0 = 2*(0.5*-508 + 0.125*-48) = 2*(-254 - 6)  = -520
      y1 = 2*(0.25*-462 + 1.0*32)   = 2*(-115.5+32) = -167
    """
    q = np.arange(1, 33, dtype=np.int8).reshape(1, 32)
    s = np.array([2.0], F32)
    w = np.array([[0x0000000F], [0x80000001]], np.uint32)
    A = np.array([[1 if k % 2 == 0 else -1 for k in range(32)]], np.int8)
    B = np.array([[3], [-2]], np.int8)
    out = o.linear(q, s, w, np.array([0.5, 0.25], F32), A, B, np.array([0.125, 1.0], F32))
    assert out["acc_s"].tolist() == [[-508, -462]]
    assert out["acc_a"].tolist() == [[-16]]
    assert out["acc_b"].tolist() == [[-48, 32]]
    assert out["y32"].tolist() == [[-520.0, -167.0]]
    assert out["y64"].tolist() == [[-520.0, -167.0]]


def pin_bruteforce(o: Oracle):
    """acc_s, acc_a, acc_b equal an int64 dense product over signs unpacked by
    numpy; y64 equals Eq. 3 evaluated literally on the dequantised input
    q(x) = s*Q in float64."""
    shapes = [(1, 32, 1, 0), (3, 64, 7, 1), (2, 96, 33, 16), (5, 768, 50, 64), (33, 128, 9, 3),
              (1, 4096, 64, 64), (2, 256, 31, 256)]
    for i, (M, K, N, r) in enumerate(shapes):
        ws, x = _case(M, K, N, r, i)
        q, s = o.quantize_act(x)
        out = o.linear(q, s, **ws)
        acc_s, acc_a, acc_b = bruteforce_int(q, ws["w_bits"], ws["A"], ws["B"])
        assert np.array_equal(out["acc_s"].astype(np.int64), acc_s), (M, K, N, r, "acc_s")
        assert np.array_equal(out["acc_a"].astype(np.int64), acc_a), (M, K, N, r, "acc_a")
        assert np.array_equal(out["acc_b"], acc_b), (M, K, N, r, "acc_b")
        qx = s.astype(np.float64)[:, None] * q.astype(np.float64)
        Sd = unpack_signs(ws["w_bits"]).astype(np.float64)
        y = ws["alpha"].astype(np.float64) * (qx @ Sd.T)
        if r:
            y = y + ws["beta"].astype(np.float64) * ((qx @ ws["A"].astype(np.float64).T) @ ws["B"].astype(np.float64).T)
        scale = np.abs(y).max() + 1e-300
        assert np.abs(out["y64"] - y).max() <= 1e-12 * scale, (M, K, N, r, "y64 vs Eq. 3")


def pin_popcount_identity(o: Oracle):
    """sum_k S_k Q_k = 2 * sum_{bit=1} Q_k - sum_k Q_k, with the masked sum
    taken over the eight two's-complement bit-planes of Q:
    sum_{bit=1} Q = sum_b c_b * popcount(w & P_b), c_b = 2^b (b<7), -128 (b=7)."""
    for i, (M, K, N) in enumerate([(1, 64, 5), (4, 2048, 17), (2, 4096, 8)]):
        ws, x = _case(M, K, N, 0, 100 + i)
        q, s = o.quantize_act(x)
        out = o.linear(q, s, ws["w_bits"], ws["alpha"], None, None, None)
        u = q.view(np.uint8)
        for m in range(M):
            planes = [np.packbits(((u[m] >> b) & 1).astype(np.uint8), bitorder="little").view("<u4")
                      for b in range(8)]
            coef = [1 << b for b in range(7)] + [-128]
            for n in range(N):
                masked = sum(c * int(np.bitwise_count(ws["w_bits"][n] & P).sum()) for c, P in zip(coef, planes))
                assert out["acc_s"][m, n] == 2 * masked - int(q[m].astype(np.int64).sum())


def pin_special_bits(o: Oracle):
    """All-ones bits -> acc_s = sum Q and (r=0) y = s*(alpha*sum Q) ("alpha times
    the row sum"); all-zeros -> -sum Q; complementing every bit negates acc_s."""
    M, K, N = 3, 256, 6
    x = S.activations(M, K, key=(92, 0))
    q, s = o.quantize_act(x)
    alpha = S.weights(K, N, 0, key=(92, 1))["alpha"]
    rs = q.astype(np.int64).sum(1)
    ones = np.full((N, K // 32), 0xFFFFFFFF, np.uint32)
    out = o.linear(q, s, ones, alpha, None, None, None)
    assert np.array_equal(out["acc_s"], np.repeat(rs[:, None], N, 1))
    exp = s[:, None] * (alpha[None, :] * rs[:, None].astype(F32))
    assert np.array_equal(out["y32"], exp.astype(F32))
    out0 = o.linear(q, s, np.zeros_like(ones), alpha, None, None, None)
    assert np.array_equal(out0["acc_s"], -np.repeat(rs[:, None], N, 1))
    w = S.weights(K, N, 0, key=(92, 2))["w_bits"]
    a = o.linear(q, s, w, alpha, None, None, None)["acc_s"]
    b = o.linear(q, s, ~w, alpha, None, None, None)["acc_s"]
    assert np.array_equal(a, -b)


def pin_permutation(o: Oracle):
    """Permuting the K axis of Q, of the signs and of A together leaves every
    accumulator unchanged."""
    M, K, N, r = 2, 192, 11, 5
    ws, x = _case(M, K, N, r, 200)
    q, s = o.quantize_act(x)
    out = o.linear(q, s, **ws)
    p = np.random.default_rng(3).permutation(K)
    Sd = unpack_signs(ws["w_bits"])
    ws2 = dict(ws, w_bits=pack_signs(Sd[:, p]), A=np.ascontiguousarray(ws["A"][:, p]))
    out2 = o.linear(np.ascontiguousarray(q[:, p]), s, **ws2)
    for k in ("acc_s", "acc_a", "acc_b"):
        assert np.array_equal(out[k], out2[k]), k


def pin_extremes(o: Oracle):
    """Closed forms at the ends of the int8 ranges: Q = 127, A = 127 ->
    acc_a = 127^2 K; B = 127 -> acc_b = 127 r 127^2 K (beyond int32);
    all-ones bits -> acc_s = 127 K.  Also with -127 operands."""
    for K, N, r in [(4096, 3, 64), (4096, 2, 256), (32, 1, 1)]:
        q = np.full((1, K), 127, np.int8)
        s = np.ones(1, F32)
        ones = np.full((N, K // 32), 0xFFFFFFFF, np.uint32)
        for sa, sb in [(1, 1), (-1, 1), (1, -1), (-1, -1)]:
            A = np.full((r, K), 127 * sa, np.int8)
            B = np.full((N, r), 127 * sb, np.int8)
            out = o.linear(q, s, ones, np.ones(N, F32), A, B, np.ones(N, F32))
            assert (out["acc_s"] == 127 * K).all()
            assert (out["acc_a"].astype(np.int64) == sa * 127 * 127 * K).all()
            assert (out["acc_b"] == sa * sb * 127 * r * 127 * 127 * K).all()


def pin_rank0(o: Oracle):
    """r = 0 is the scaffold alone: y = s*(alpha*acc_s).  A = 0 (or B = 0)
    with r > 0 gives acc_b = 0 and the same y values."""
    M, K, N, r = 3, 512, 40, 16
    ws, x = _case(M, K, N, r, 300)
    q, s = o.quantize_act(x)
    base = o.linear(q, s, ws["w_bits"], ws["alpha"], None, None, None)
    exp = (s[:, None] * (ws["alpha"][None, :] * base["acc_s"].astype(F32))).astype(F32)
    assert np.array_equal(base["y32"], exp)
    assert np.array_equal(base["y64"], s[:, None].astype(np.float64)
                          * (ws["alpha"][None, :].astype(np.float64) * base["acc_s"]))
    for zA in (True, False):
        A = np.zeros_like(ws["A"]) if zA else ws["A"]
        B = ws["B"] if zA else np.zeros_like(ws["B"])
        out = o.linear(q, s, ws["w_bits"], ws["alpha"], A, B, ws["beta"])
        assert not out["acc_b"].any()
        assert np.array_equal(out["acc_s"], base["acc_s"])
        assert (out["y32"] == base["y32"]).all()


def pin_y32_order(o: Oracle):
    """y32 is the fp32 evaluation of y64: within a few fp32 roundings of it,
    and equal to the op-by-op fp32 sequence on the exact accumulators."""
    for i, (M, K, N, r) in enumerate([(2, 2048, 300, 64), (1, 768, 3352, 16), (3, 4096, 100, 64)]):
        for bs in (1.0, 1.8e-5):
            ws, x = _case(M, K, N, r, 400 + i, beta_scale=bs)
            q, s = o.quantize_act(x)
            out = o.linear(q, s, **ws)
            y64 = out["y64"]
            assert np.abs(out["y32"] - y64).max() <= 1e-6 * np.abs(y64).max()
            acc_s, acc_a, acc_b = bruteforce_int(q, ws["w_bits"], ws["A"], ws["B"])
            u = ws["alpha"][None, :] * acc_s.astype(F32)
            v = ws["beta"][None, :] * acc_b.astype(F32)
            assert np.array_equal(out["y32"], (s[:, None] * (u + v)).astype(F32))


def pin_chain(o: Oracle):
    """The chain: linear 0 reads (Q0, s0); linear l reads the quantised
    prefix y_{l-1}[:, :K_l] with s fixed to 1/127.  Checked against a chain
    built from brute-force integer products and the quantiser pinned above;
    the sweep's magnitudes stay bounded over 96 linears."""
    shapes = [(64, 96), (96, 64), (64, 160), (128, 64)]
    layers = [S.weights(K, N, 4, key=(93, i, K, N)) for i, (K, N) in enumerate(shapes)]
    x = S.activations(2, 64, key=(93, 9))
    q0, s0 = o.quantize_act(x)
    ys, qs = o.chain(layers, q0, s0)
    q, s = q0, s0
    for l, ly in enumerate(layers):
        if l:
            q, _ = o.quantize_act(ys[l - 1].astype(F32), K=shapes[l][0])
            s = np.full(2, F32(1.0) / F32(127.0), F32)
        assert np.array_equal(qs[l], q), l
        acc_s, _, acc_b = bruteforce_int(q, ly["w_bits"], ly["A"], ly["B"])
        y = (s[:, None] * (ly["alpha"][None, :] * acc_s.astype(F32) + ly["beta"][None, :] * acc_b.astype(F32))).astype(F32)
        assert np.array_equal(ys[l], y), l
    # bounded over a long chain at the 1.3B shapes (short K keeps it quick)
    shapes = [(256, 512), (512, 256)] * 48
    layers = [S.weights(K, N, 8, key=(94, i, K, N)) for i, (K, N) in enumerate(shapes)]
    q0, s0 = o.quantize_act(S.activations(1, 256, key=(94, 0)))
    ys, _ = o.chain(layers, q0, s0)
    for y in ys:
        assert np.isfinite(y).all() and 1e-3 < np.abs(y).max() < 1e6


def pin_paper_sizes(o: Oracle):
    """Table 1: the 48-layer scaffold at 1 bit per weight is "155 MB" (56% of
    278 MB) and the int8 r=16 LoRA "12 MB" -- computed from the byte sizes of
    the arrays in the layout the library takes."""
    facts = json.load(open(os.path.join(GOLDEN, "paper_facts.json")))
    t1 = facts["model_size_table"]
    sign_bytes = lora_bytes = 0
    for K, N in S.sweep_shapes(facts["model_shape"]["n_layers"]):
        sign_bytes += N * (K // 32) * np.dtype(np.uint32).itemsize
        lora_bytes += (16 * K + N * 16) * np.dtype(np.int8).itemsize
    assert sign_bytes == 154_927_104
    assert round(sign_bytes / 1e6) == t1["scaffold_48_layers_in_out_proj_1bit_MB"]
    assert round(100 * sign_bytes / 1e6 / t1["total_MB"]) == t1["scaffold_fraction_percent"]
    # one byte per LoRA value: 12.83e6 bytes; the table prints "12 MB" (its
    # rounding/unit for this row is not stated), so allow 10%
    assert abs(lora_bytes / 1e6 - t1["lora_48_layers_r16_int8_MB"]) <= 0.1 * t1["lora_48_layers_r16_int8_MB"]
    ks = facts["cpu_kernel"]
    assert 2048 // ks["weights_per_64bit_load"] == ks["vpdpbusd_per_2048_row"]
    # a sign bit per weight: an all-shapes weight set has K*N/8 sign bytes
    ws = S.weights(2048, 8512, 16, key=(95,))
    assert ws["w_bits"].nbytes * 8 == 2048 * 8512
    # the tied int8 embedding / LM head: one byte per entry of the
    # 50,280 x 2048 table is "103 MB", 37% of the 278 MB model
    # in_proj's width: [z | x | B | C | dt] of a Mamba-2 mixer with
    # d_inner = 2 d_model, heads of 64 and Table 12's d_state 128
    ms = facts["model_shape"]
    dm = S.mamba_dims(ms["d_model"], ms["d_state"], 64)
    assert dm["ld"] == 2 * dm["d_inner"] + 2 * ms["d_state"] + dm["nheads"] == S.IN_PROJ_1P3B[1]
    emb = 50_280 * facts["model_shape"]["d_model"] * np.dtype(np.int8).itemsize
    assert round(emb / 1e6) == t1["embedding_lm_head_int8_MB"]
    assert round(100 * emb / 1e6 / t1["total_MB"]) == 37


# --------------------------------------------------------------------------
# tied int8 embedding / LM head
# --------------------------------------------------------------------------
def pin_embed_lm_hand(o: Oracle):
    """Hand-derived: E = [[1, 2], [3, -4], [5, 6]], row scales (0.5, 2, 1)."""
    E = np.array([[1, 2], [3, -4], [5, 6]], np.int8)
    sc = np.array([0.5, 2.0, 1.0], F32)
    x = o.embed_gather(E, sc, np.array([1, 0, 2], np.int32))
    assert np.array_equal(x, np.array([[6, -8], [0.5, 1], [5, 6]], F32))
    q = np.array([[1, 1], [2, -1]], np.int8)
    s = np.array([0.25, 1.0], F32)
    acc, logits = o.lm_head(q, s, E, sc)
    assert np.array_equal(acc, np.array([[3, -1, 11], [0, 10, 4]], np.int32))
    assert np.array_equal(logits, np.array([[0.375, -0.5, 2.75], [0.0, 20.0, 4.0]], F32))


def _lm_case(M, V, d, seed):
    rng = np.random.default_rng(seed)
    E = rng.integers(-127, 128, (V, d), dtype=np.int8)
    sc = rng.uniform(1e-3, 2e-2, V).astype(F32)
    q, s = o_quant(M, d, seed)
    return E, sc, q, s


def o_quant(M, d, seed):
    """Codes and scales from an independent quantiser written here (the
    definition: s = a/127, Q = rint(x * (127/a)), fp32 each step)."""
    x = S.activations(M, d, key=(96, seed)).astype(F32)
    a = np.abs(x).max(axis=1).astype(F32)
    s = (a / F32(127)).astype(F32)
    inv = (F32(127) / a).astype(F32)
    q = np.clip(np.rint((x * inv[:, None]).astype(F32)), -127, 127).astype(np.int8)
    return q, s


def pin_lm_head_bruteforce(o: Oracle):
    """acc by an int64 matrix product; logits in the stated fp32 order,
    element by element with numpy float32 scalars (one rounding each)."""
    E, sc, q, s = _lm_case(3, 37, 96, 1)
    acc, logits = o.lm_head(q, s, E, sc)
    ref = q.astype(np.int64) @ E.astype(np.int64).T
    assert np.array_equal(acc, ref.astype(np.int32))
    for m in range(3):
        for v in range(37):
            t = F32(sc[v]) * F32(ref[m, v])
            assert logits[m, v] == F32(s[m]) * t, (m, v)
    # (float)acc rounds to nearest-even above 2^24: a row of all 127 against
    # codes of all 127 gives 127^2 * 1056 = 17,032,224 (even, exact) and
    # with one code 126 gives 17,032,097, which fp32 rounds to 17,032,096
    E2 = np.full((2, 1056), 127, np.int8)
    q2 = np.full((1, 1056), 127, np.int8)
    q2[0, 0] = 126
    acc2, lg2 = o.lm_head(q2, np.ones(1, F32), E2, np.ones(2, F32))
    assert acc2[0, 0] == 17_032_097 and lg2[0, 0] == F32(17_032_096)


def pin_lm_head_closed_forms(o: Oracle):
    """All-ones rows with unit scale give the row sum of the codes; identity
    rows give the codes themselves; the scale of row v scales only logit v."""
    _, _, q, s = _lm_case(2, 1, 64, 2)
    acc, _ = o.lm_head(q, s, np.ones((3, 64), np.int8), np.ones(3, F32))
    assert np.array_equal(acc, np.repeat(q.astype(np.int64).sum(axis=1, keepdims=True), 3, axis=1))
    acc, logits = o.lm_head(q, s, np.eye(64, dtype=np.int8), np.ones(64, F32))
    assert np.array_equal(acc, q.astype(np.int32))
    assert np.array_equal(logits, (s[:, None] * q.astype(F32)).astype(F32))
    E, sc, q, s = _lm_case(2, 11, 32, 3)
    _, l1 = o.lm_head(q, s, E, sc)
    sc2 = sc.copy()
    sc2[4] *= F32(2)
    _, l2 = o.lm_head(q, s, E, sc2)
    assert np.array_equal(np.delete(l1, 4, axis=1), np.delete(l2, 4, axis=1))
    assert np.array_equal(l2[:, 4], (F32(2) * l1[:, 4]).astype(F32))


def pin_embed_gather_bruteforce(o: Oracle):
    """Each gathered value is one fp32 product scale[t] * E[t, k]; ids out of
    range are refused."""
    E, sc, _, _ = _lm_case(1, 29, 64, 4)
    tok = np.array([28, 0, 5, 5], np.int32)
    x = o.embed_gather(E, sc, tok)
    for m, t in enumerate(tok):
        for k in range(64):
            assert x[m, k] == F32(sc[t]) * F32(E[t, k])
    for bad in ([29], [-1]):
        try:
            o.embed_gather(E, sc, np.array(bad, np.int32))
        except OracleError as e:
            assert e.status == 2
        else:
            raise AssertionError("an out-of-range token id was accepted")


# --------------------------------------------------------------------------
# int4 LoRA factors
# --------------------------------------------------------------------------
def _unpack_np(packed: np.ndarray, n: int) -> np.ndarray:
    """Independent route: numpy shifts and masks, then two's complement."""
    p = packed.astype(np.uint8).ravel()
    nib = np.empty(2 * p.size, np.int16)
    nib[0::2] = p & 0x0F
    nib[1::2] = p >> 4
    return np.where(nib >= 8, nib - 16, nib)[:n].astype(np.int8)


def pin_int4(o: Oracle):
    """Hand-derived nibbles, every byte value against numpy's route, and the
    int4 linear equal to brute force on the unpacked factors."""
    # 0x2F: low nibble 0xF = -1, high 0x2 = 2; 0x87: 7 then -8; 0x80: 0, -8
    assert o.unpack_int4(np.array([0x2F, 0x87, 0x80], np.uint8), 6).tolist() == [-1, 2, 7, -8, 0, -8]
    allb = np.arange(256, dtype=np.uint8)
    assert np.array_equal(o.unpack_int4(allb, 512), _unpack_np(allb, 512))
    assert o.unpack_int4(np.array([0x7F], np.uint8), 1).tolist() == [-1]        # odd count
    ws = S.weights_i4(96, 37, 6, key=(96, 1))
    x = S.activations(3, 96, key=(96, 2))
    q, s = o.quantize_act(x)
    ref = o.linear_i4(q, s, **ws)
    A = _unpack_np(ws["A4"], 6 * 96).reshape(6, 96)
    B = _unpack_np(ws["B4"], 37 * 6).reshape(37, 6)
    acc_s, acc_a, acc_b = bruteforce_int(q, ws["w_bits"], A, B)
    assert np.array_equal(ref["acc_s"], acc_s) and np.array_equal(ref["acc_a"], acc_a)
    assert np.array_equal(ref["acc_b"], acc_b)


# --------------------------------------------------------------------------
# Mamba-2 decode step around the linears
# --------------------------------------------------------------------------
def _silu64(v):
    """silu through scipy's logistic function (a library routine)."""
    from scipy.special import expit
    v = np.asarray(v, np.float64)
    return v * expit(v)


def pin_rmsnorm(o: Oracle):
    """Hand case, the normalisation property, scale invariance, the weight
    acting per channel, the role of eps and the residual add."""
    # u = [3, 4, 0, 0], eps = 0: mean square 25/4, r = 0.4 (rounded to fp32),
    # o = [1.2, 1.6, 0, 0]; Q = rint(1.2 / 1.6 * 127) = rint(95.25) = 95
    u = np.array([[3, 4, 0, 0]], F32)
    _, on, q, s = o.add_rmsnorm_quant(u, np.ones(4, F32), 0.0)
    assert np.allclose(on[0], [1.2, 1.6, 0, 0], rtol=1e-7, atol=0)
    assert q[0].tolist() == [95, 127, 0, 0]
    assert abs(float(s[0]) - 1.6 / 127) <= 1e-7 * 1.6 / 127
    # eps = 0, unit weight: mean(o^2) = 1 for any row
    x = S.residual(3, 512, key=(98,))
    one = np.ones(512, F32)
    _, on, q, s = o.add_rmsnorm_quant(x, one, 0.0)
    assert np.allclose((on.astype(np.float64) ** 2).mean(axis=1), 1.0, rtol=0, atol=1e-6)
    # eps = 0: scaling the row by a power of two changes nothing
    _, o2, q2, s2 = o.add_rmsnorm_quant(x * F32(8), one, 0.0)
    assert np.array_equal(o2, on) and np.array_equal(q2, q) and np.array_equal(s2, s)
    # the weight scales each channel of the unit-weight output
    w = np.random.default_rng(99).uniform(0.5, 2.0, 512).astype(F32)
    _, ow, _, _ = o.add_rmsnorm_quant(x, w, 0.0)
    assert np.array_equal(ow, (on * w).astype(F32))
    # eps equal to the mean square halves it into 1/sqrt(2 m): a row of 2s
    # with eps = 4 gives o = 2 / sqrt(8) = 1/sqrt(2)
    _, on, _, _ = o.add_rmsnorm_quant(np.full((1, 64), 2.0, F32), np.ones(64, F32), 4.0)
    assert np.allclose(on, 2 ** -0.5, rtol=2e-7, atol=0)
    # residual: u + (-u) is a zero row (Q = 0, s = 0); u_out is the sum
    u_out, on, q, s = o.add_rmsnorm_quant(x, one, 1e-5, delta=-x)
    assert not u_out.any() and not q.any() and not s.any() and not on.any()
    d = S.residual(3, 512, key=(100,))
    u_out, _, _, _ = o.add_rmsnorm_quant(x, one, 1e-5, delta=d)
    assert np.array_equal(u_out, (x + d).astype(F32))


# small mixer for the step pins: d_inner 64, N 8, P 16 -> 4 heads, conv_dim 80
_DI, _N, _P = 64, 8, 16


def _small_params(seed, **over):
    p = S.mamba_params(_DI // 2, d_state=_N, headdim=_P, key=(101, seed))
    p.update(over)
    return p


def _zero_state(M):
    H = _DI // _P
    return np.zeros((M, _DI + 2 * _N, 4), F32), np.zeros((M, H, _P, _N), F32)


def _step(o, zx, cs, hs, p):
    return o.ssm_step(zx, cs, hs, p["conv_w"], p["conv_b"], p["dt_bias"], p["A_log"], p["D"], _DI, _N, _P)


def pin_conv_step(o: Oracle):
    """An impulse through the shift register: at step t after it, channel c
    shows silu(w[c][3 - t]); it is gone after 4 steps.  A constant input
    shows silu(sum_j w[c][j] + b[c]) once the register is full."""
    p = _small_params(0, conv_b=np.zeros(_DI + 2 * _N, F32))
    ld = S.mamba_dims(_DI // 2, _N, _P)["ld"]
    cs, hs = _zero_state(1)
    chans = [5, _DI + 3, _DI + _N + 7]             # an x, a B and a C channel
    for t in range(6):
        zx = np.zeros((1, ld), F32)
        if t == 0:
            zx[0, _DI + np.array(chans)] = 1.0
        _, xbc, cs, hs = _step(o, zx, cs, hs, p)
        want = np.zeros(_DI + 2 * _N)
        if t < 4:
            for c in chans:
                want[c] = _silu64(p["conv_w"][c, 3 - t])
        assert np.allclose(xbc[0], want, rtol=1e-6, atol=0), t
    assert not cs.any()
    # constant input 1 with a bias: silu(sum_j w[c][j] + b[c]) from step 3 on
    p = _small_params(1)
    cs, hs = _zero_state(1)
    zx = np.zeros((1, ld), F32)
    zx[0, _DI:_DI + _DI + 2 * _N] = 1.0
    for _ in range(4):
        _, xbc, cs, hs = _step(o, zx, cs, hs, p)
    want = _silu64(p["conv_w"].astype(np.float64).sum(axis=1) + p["conv_b"])
    assert np.allclose(xbc[0], want, rtol=1e-6, atol=1e-7)


def _ident_conv(p):
    """Taps [0, 0, 0, 1] and no bias: the conv output is silu(newest input)."""
    w = np.zeros((_DI + 2 * _N, 4), F32)
    w[:, 3] = 1.0
    p = dict(p)
    p["conv_w"], p["conv_b"] = w, np.zeros(_DI + 2 * _N, F32)
    return p


def pin_ssm_step(o: Oracle):
    """Closed forms of the recurrence h = h dA + (x dt) B, y = C.h + D x:
    a memoryless head (dA = 0), pure decay over 3 steps, the geometric sum
    from a zero state, the D skip, and head independence."""
    H = _DI // _P
    ld = S.mamba_dims(_DI // 2, _N, _P)["ld"]
    dt_off = _DI + _DI + 2 * _N
    rng = np.random.default_rng(102)
    # (a) dt above the softplus threshold is taken as is; A_log = 30 makes
    # dt * A far below exp's range, so dA = 0 and the state is (x dt) B
    p = _ident_conv(_small_params(2, dt_bias=np.full(H, 25.0, F32), A_log=np.full(H, 30.0, F32)))
    zx = rng.standard_normal((2, ld)).astype(F32)
    cs = S.mamba_state(2, _DI // 2, _N, _P, key=(103,))
    y, xbc, _, hs = _step(o, zx, cs["conv_state"], cs["ssm_state"], p)
    dt = (zx[:, dt_off:dt_off + H] + F32(25.0)).astype(np.float64)              # [M, H]
    x = xbc[:, :_DI].astype(np.float64).reshape(2, H, _P)
    B = xbc[:, _DI:_DI + _N].astype(np.float64)
    C = xbc[:, _DI + _N:].astype(np.float64)
    h_want = dt[:, :, None, None] * x[:, :, :, None] * B[:, None, None, :]
    assert np.allclose(hs, h_want, rtol=3e-7, atol=0)
    y_want = (h_want * C[:, None, None, :]).sum(axis=3) + p["D"][None, :, None] * x
    bound = 1e-6 * (np.abs(h_want * C[:, None, None, :]).sum(axis=3) + np.abs(p["D"][None, :, None] * x))
    assert np.all(np.abs(y.reshape(2, H, _P) - y_want) <= bound)
    # (b) x = 0 (silu(0)): pure decay, h_3 = h_0 exp(3 dt A) with
    # dt = softplus(v) from numpy's logaddexp
    p = _ident_conv(_small_params(3))
    h0 = S.mamba_state(1, _DI // 2, _N, _P, key=(104,))["ssm_state"]
    zx = np.zeros((1, ld), F32)
    zx[0, _DI + _DI:_DI + _DI + 2 * _N] = rng.standard_normal(2 * _N)            # B and C inputs
    zx[0, dt_off:] = rng.standard_normal(H)
    hs = h0
    cs = np.zeros((1, _DI + 2 * _N, 4), F32)
    for _ in range(3):
        y, xbc, cs, hs = _step(o, zx, cs, hs, p)
    sp = np.logaddexp(0.0, (zx[0, dt_off:] + p["dt_bias"]).astype(np.float64))
    A = -np.exp(p["A_log"].astype(np.float64))
    dec = np.exp(3 * sp * A)
    h_want = h0[0].astype(np.float64) * dec[:, None, None]
    assert np.allclose(hs[0], h_want, rtol=2e-6, atol=1e-30)
    C = xbc[0, _DI + _N:].astype(np.float64)
    assert np.allclose(y[0].reshape(H, _P), (h_want * C).sum(axis=2), rtol=1e-5, atol=1e-6)
    # (c) from a zero state with a constant input: h_T = dt x B (1 - dA^T) / (1 - dA)
    p = _ident_conv(_small_params(4))
    zx = np.zeros((1, ld), F32)
    zx[0, _DI:] = rng.standard_normal(ld - _DI)
    cs, hs = _zero_state(1)
    T = 5
    for _ in range(T):
        y, xbc, cs, hs = _step(o, zx, cs, hs, p)
    dt = np.logaddexp(0.0, (zx[0, dt_off:] + p["dt_bias"]).astype(np.float64))
    dA = np.exp(dt * -np.exp(p["A_log"].astype(np.float64)))
    x = xbc[0, :_DI].astype(np.float64).reshape(H, _P)
    B = xbc[0, _DI:_DI + _N].astype(np.float64)
    C = xbc[0, _DI + _N:].astype(np.float64)
    geo = (1 - dA ** T) / (1 - dA)
    h_want = (dt * geo)[:, None, None] * x[:, :, None] * B[None, None, :]
    assert np.allclose(hs[0], h_want, rtol=1e-5, atol=1e-12)
    y_want = (h_want * C).sum(axis=2) + p["D"][:, None] * x
    assert np.allclose(y[0].reshape(H, _P), y_want, rtol=1e-5, atol=1e-6)
    # (d) B = 0 and a zero state: y is the D skip alone, D x rounded once
    zx[0, _DI + _DI:_DI + _DI + _N] = 0.0
    cs, hs = _zero_state(1)
    y, xbc, _, hs = _step(o, zx, cs, hs, p)
    assert not hs.any()
    x = xbc[0, :_DI].reshape(H, _P)
    assert np.array_equal(y[0].reshape(H, _P), (p["D"][:, None] * x).astype(F32))
    # (e) heads are independent: permuting everything per head permutes y
    p = _small_params(5)
    st = S.mamba_state(1, _DI // 2, _N, _P, key=(105,))
    zx = rng.standard_normal((1, ld)).astype(F32)
    y, _, _, hs = _step(o, zx, st["conv_state"], st["ssm_state"], p)
    perm = np.array([2, 0, 3, 1])
    ch = (perm[:, None] * _P + np.arange(_P)[None, :]).ravel()                    # x channels
    cperm = np.concatenate([ch, np.arange(_DI, _DI + 2 * _N)])
    p2 = dict(p)
    p2["conv_w"], p2["conv_b"] = p["conv_w"][cperm], p["conv_b"][cperm]
    for k in ("dt_bias", "A_log", "D"):
        p2[k] = p[k][perm]
    zx2 = zx.copy()
    zx2[0, _DI:_DI + _DI + 2 * _N] = zx[0, _DI + cperm]
    zx2[0, dt_off:] = zx[0, dt_off + perm]
    zx2[0, :_DI] = zx[0, ch]
    y2, _, _, hs2 = _step(o, zx2, st["conv_state"][:, cperm], st["ssm_state"][:, perm], p2)
    assert np.array_equal(y2[0], y[0][ch]) and np.array_equal(hs2[0], hs[0][perm])


def pin_gate_norm(o: Oracle):
    """Gate before norm (Table 12): norm(y silu(z)).  A constant row
    normalises to 1 whatever the gate, so s = 1/127; an identity gate
    (silu(30) = 30 in fp32) equals the plain norm of 30 y; silu(0) = 0
    zeroes a channel; the output has unit mean square."""
    one = np.ones(64, F32)
    _, q, s = o.gate_norm_quant(np.full((1, 64), 3.0, F32), np.full((1, 64), 0.7, F32), one, 0.0)
    assert np.all(q == 127) and abs(float(s[0]) * 127 - 1.0) <= 2e-7
    y = S.residual(2, 256, key=(106,))
    w = np.random.default_rng(107).uniform(0.8, 1.2, 256).astype(F32)
    og, qg, sg = o.gate_norm_quant(y, np.full((2, 256), 30.0, F32), w, 1e-5)
    _, on, qn, sn = o.add_rmsnorm_quant((y * F32(30.0)).astype(F32), w, 1e-5)
    assert np.array_equal(og, on) and np.array_equal(qg, qn) and np.array_equal(sg, sn)
    z = np.random.default_rng(108).standard_normal((2, 256)).astype(F32)
    z[:, ::7] = 0.0
    og, qg, _ = o.gate_norm_quant(y, z, np.ones(256, F32), 0.0)
    assert not og[:, ::7].any() and not qg[:, ::7].any()
    assert np.allclose((og.astype(np.float64) ** 2).mean(axis=1), 1.0, rtol=0, atol=1e-6)
    _, q0, s0 = o.gate_norm_quant(np.zeros((1, 64), F32), np.ones((1, 64), F32), one, 1e-5)
    assert not q0.any() and not s0.any()


def pin_validation(o: Oracle):
    """Shapes outside the contract are refused with the shape status."""
    q = np.zeros(64, np.int8)
    one = np.ones(4, F32)
    w = np.zeros(8, np.uint32)
    p = lambda a: a.ctypes.data
    f = o.lib.dfssm_ref_scaffold_lora_linear
    for (M, K, N, r) in [(1, 48, 1, 0), (1, 0, 1, 0), (-1, 32, 1, 0), (1, 32, -1, 0), (1, 32, 1, 257), (1, 32, 1, -1)]:
        assert f(p(q), p(one), M, K, N, r, p(w), p(one), p(q), p(q), p(one), None, None, None, None, None) == 2
    assert o.lib.dfssm_ref_quantize_act(p(one), 1, 1, 4, 3, p(q), p(one)) == 2  # ldx < K


ALL_PINS = [pin_f16_decode, pin_quantize_hand_cases, pin_quantize_properties, pin_hand_linear,
            pin_bruteforce, pin_popcount_identity, pin_special_bits, pin_permutation, pin_extremes,
            pin_rank0, pin_y32_order, pin_chain, pin_paper_sizes, pin_embed_lm_hand, pin_lm_head_bruteforce,
            pin_lm_head_closed_forms, pin_embed_gather_bruteforce, pin_rmsnorm, pin_conv_step, pin_ssm_step,
            pin_gate_norm, pin_int4, pin_validation]
