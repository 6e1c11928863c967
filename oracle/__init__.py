"""CPU oracle for the DF-SSM scaffold + int8 LoRA linear (test infrastructure).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It wraps the plain C implementation in dfssm_ref.c
(built with gcc, no GPU code, no code shared with the HIP library) in numpy
helpers.  See dfssm_ref.h for the definitions it follows (Sec. 3.2 Eq. 3,
Sec. 3.3 / Table 1, Sec. 4.1 of the paper).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "dfssm_ref.c")
LIB = os.path.join(HERE, "libdfssm_ref.so")

OK, ERR_NULL, ERR_SHAPE, ERR_NONFINITE = 0, 1, 2, 7
F16, F32 = 0, 1


def build(src: str = SRC, out: str = LIB, extra: Sequence[str] = (), openmp: bool = True) -> str:
    """Compile the oracle with gcc: -O2, no contraction, no fast-math."""
    cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-Werror", "-I", HERE]
    if openmp:
        cmd.append("-fopenmp")
    cmd += list(extra) + [src, "-o", out, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """numpy front end over one build of the C oracle (a path to a .so)."""

    def __init__(self, path: str = LIB):
        if not os.path.exists(path):
            build(out=path)
        self.path = path
        lib = ctypes.CDLL(path)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        lib.dfssm_ref_f16_to_f32.argtypes = [ctypes.c_uint16]
        lib.dfssm_ref_f16_to_f32.restype = ctypes.c_float
        lib.dfssm_ref_quantize_act.argtypes = [vp, i32, i64, i64, i64, vp, vp]
        lib.dfssm_ref_quantize_act.restype = i32
        lib.dfssm_ref_scaffold_lora_linear.argtypes = [vp, vp, i64, i64, i64, i64, vp, vp, vp, vp,
                                                       vp, vp, vp, vp, vp, vp]
        lib.dfssm_ref_scaffold_lora_linear.restype = i32
        lib.dfssm_ref_chain.argtypes = [i32, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.dfssm_ref_chain.restype = i32
        lib.dfssm_ref_threads.restype = i32
        lib.dfssm_ref_set_threads.argtypes = [i32]
        lib.dfssm_ref_set_threads.restype = None
        lib.dfssm_ref_embed_gather.argtypes = [vp, vp, i64, i64, vp, i64, vp]
        lib.dfssm_ref_embed_gather.restype = i32
        lib.dfssm_ref_lm_head.argtypes = [vp, vp, i64, i64, vp, vp, i64, vp, vp]
        lib.dfssm_ref_lm_head.restype = i32
        f32 = ctypes.c_float
        lib.dfssm_ref_unpack_int4.argtypes = [vp, i64, vp]
        lib.dfssm_ref_unpack_int4.restype = i32
        lib.dfssm_ref_add_rmsnorm_quant.argtypes = [vp, vp, vp, f32, i64, i64, vp, vp, vp, vp]
        lib.dfssm_ref_add_rmsnorm_quant.restype = i32
        lib.dfssm_ref_ssm_step.argtypes = [vp, i64, i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.dfssm_ref_ssm_step.restype = i32
        lib.dfssm_ref_gate_norm_quant.argtypes = [vp, vp, i64, vp, f32, i64, i64, vp, vp, vp]
        lib.dfssm_ref_gate_norm_quant.restype = i32
        self.lib = lib

    # -- activation quantisation ------------------------------------------------
    def f16_to_f32(self, h: int) -> float:
        return self.lib.dfssm_ref_f16_to_f32(int(h))

    def quantize_act(self, x: np.ndarray, K: Optional[int] = None):
        """x: [M, ldx] float16 or float32; quantises the first K columns.
        Returns (Q int8 [M,K], s float32 [M]); raises on a status error."""
        x = np.ascontiguousarray(x)
        if x.ndim != 2:
            raise ValueError("x must be 2-D")
        M, ldx = x.shape
        K = ldx if K is None else K
        dt = {np.dtype(np.float16): F16, np.dtype(np.float32): F32}[x.dtype]
        q = np.zeros((M, K), np.int8)
        s = np.zeros((M,), np.float32)
        st = self.lib.dfssm_ref_quantize_act(_p(x), dt, M, K, ldx, _p(q), _p(s))
        if st != OK:
            raise OracleError(st)
        return q, s

    # -- the linear -----------------------------------------------------------------
    def linear(self, q, s, w_bits, alpha, A, B, beta):
        """Returns dict with acc_s (int32 [M,N]), acc_a (int32 [M,r]),
        acc_b (int64 [M,N]), y32 (float32 [M,N]), y64 (float64 [M,N])."""
        q = np.ascontiguousarray(q, np.int8)
        s = np.ascontiguousarray(s, np.float32)
        w_bits = np.ascontiguousarray(w_bits, np.uint32)
        alpha = np.ascontiguousarray(alpha, np.float32)
        M, K = q.shape
        N = w_bits.shape[0]
        if w_bits.shape[1] * 32 != K:
            raise ValueError("w_bits must be [N, K/32]")
        r = 0 if A is None else A.shape[0]
        if r > 0:
            A = np.ascontiguousarray(A, np.int8)
            B = np.ascontiguousarray(B, np.int8)
            beta = np.ascontiguousarray(beta, np.float32)
        else:
            A = B = beta = None
        out = dict(acc_s=np.zeros((M, N), np.int32), acc_a=np.zeros((M, max(r, 0)), np.int32),
                   acc_b=np.zeros((M, N), np.int64), y32=np.zeros((M, N), np.float32),
                   y64=np.zeros((M, N), np.float64))
        st = self.lib.dfssm_ref_scaffold_lora_linear(
            _p(q), _p(s), M, K, N, r, _p(w_bits), _p(alpha), _p(A), _p(B), _p(beta),
            _p(out["acc_s"]), _p(out["acc_a"]) if r > 0 else None, _p(out["acc_b"]),
            _p(out["y32"]), _p(out["y64"]))
        if st != OK:
            raise OracleError(st)
        return out

    # -- the chain ------------------------------------------------------------------
    def chain(self, layers, q0, s0):
        """layers: sequence of dicts with w_bits, alpha, A, B, beta.
        Returns (list of y32 [M,N_l], list of Q [M,K_l])."""
        q0 = np.ascontiguousarray(q0, np.int8)
        s0 = np.ascontiguousarray(s0, np.float32)
        M = q0.shape[0]
        L = len(layers)
        Ks = np.array([ly["w_bits"].shape[1] * 32 for ly in layers], np.int64)
        Ns = np.array([ly["w_bits"].shape[0] for ly in layers], np.int64)
        rs = np.array([0 if ly.get("A") is None else ly["A"].shape[0] for ly in layers], np.int64)
        keep = []

        def arr(name, dtype):
            ptrs = (ctypes.c_void_p * L)()
            for i, ly in enumerate(layers):
                a = ly.get(name)
                if a is None or (name in ("A", "B", "beta") and rs[i] == 0):
                    ptrs[i] = None
                    continue
                a = np.ascontiguousarray(a, dtype)
                keep.append(a)
                ptrs[i] = a.ctypes.data
            return ptrs

        pw, pa, pA, pB, pb = (arr("w_bits", np.uint32), arr("alpha", np.float32),
                              arr("A", np.int8), arr("B", np.int8), arr("beta", np.float32))
        y_all = np.zeros(int((M * Ns).sum()), np.float32)
        q_all = np.zeros(int((M * Ks).sum()), np.int8)
        st = self.lib.dfssm_ref_chain(L, M, _p(Ks), _p(Ns), _p(rs), pw, pa, pA, pB, pb,
                                      _p(q0), _p(s0), _p(y_all), _p(q_all))
        if st != OK:
            raise OracleError(st)
        ys, qs, yo, qo = [], [], 0, 0
        for l in range(L):
            ys.append(y_all[yo:yo + M * Ns[l]].reshape(M, Ns[l]))
            qs.append(q_all[qo:qo + M * Ks[l]].reshape(M, Ks[l]))
            yo += M * Ns[l]
            qo += M * Ks[l]
        return ys, qs

    # -- tied int8 embedding / LM head -------------------------------------------
    def embed_gather(self, E, scale, tok):
        """x [M,d] float32 = scale[tok] * E[tok, :]."""
        E = np.ascontiguousarray(E, np.int8)
        scale = np.ascontiguousarray(scale, np.float32)
        tok = np.ascontiguousarray(tok, np.int32)
        V, d = E.shape
        M = tok.shape[0]
        x = np.zeros((M, d), np.float32)
        st = self.lib.dfssm_ref_embed_gather(_p(E), _p(scale), V, d, _p(tok), M, _p(x))
        if st != OK:
            raise OracleError(st)
        return x

    def lm_head(self, q, s, E, scale):
        """Returns (acc int32 [M,V], logits float32 [M,V])."""
        q = np.ascontiguousarray(q, np.int8)
        s = np.ascontiguousarray(s, np.float32)
        E = np.ascontiguousarray(E, np.int8)
        scale = np.ascontiguousarray(scale, np.float32)
        M, d = q.shape
        V = E.shape[0]
        if E.shape[1] != d:
            raise ValueError("E must be [V, d]")
        acc = np.zeros((M, V), np.int32)
        logits = np.zeros((M, V), np.float32)
        st = self.lib.dfssm_ref_lm_head(_p(q), _p(s), M, d, _p(E), _p(scale), V, _p(acc), _p(logits))
        if st != OK:
            raise OracleError(st)
        return acc, logits

    # ---- int4 LoRA factors --------------------------------------------------
    def unpack_int4(self, packed, n: int):
        """n int8 values from two's-complement nibbles, low nibble first."""
        p = np.ascontiguousarray(packed, np.uint8).ravel()
        if p.size * 2 < n:
            raise ValueError("too few packed bytes")
        out = np.zeros(n, np.int8)
        st = self.lib.dfssm_ref_unpack_int4(_p(p), n, _p(out))
        if st != OK:
            raise OracleError(st)
        return out

    def linear_i4(self, q, s, w_bits, alpha, A4, B4, beta):
        """The linear with int4 LoRA factors A4 [r][K/2], B4 [N][r/2] bytes:
        the int8 linear on the unpacked factors."""
        K = q.shape[1]
        N = w_bits.shape[0]
        if A4 is None or A4.size == 0:
            return self.linear(q, s, w_bits, alpha, None, None, None)
        r = A4.shape[0]
        A = self.unpack_int4(A4, r * K).reshape(r, K)
        B = self.unpack_int4(B4, N * r).reshape(N, r)
        return self.linear(q, s, w_bits, alpha, A, B, beta)

    def chain_i4(self, layers, q0, s0):
        """The chain whose layers carry int4 LoRA factors (A4, B4; or int8
        A, B): the chain on the unpacked factors, as linear_i4 (Table 4
        keeps the LoRA arithmetic and only narrows the stored factors)."""
        out = []
        for ly in layers:
            if ly.get("A4") is None:
                out.append(ly)
                continue
            K, N, r = ly["w_bits"].shape[1] * 32, ly["w_bits"].shape[0], ly["A4"].shape[0]
            out.append(dict(w_bits=ly["w_bits"], alpha=ly["alpha"], beta=ly["beta"],
                            A=self.unpack_int4(ly["A4"], r * K).reshape(r, K),
                            B=self.unpack_int4(ly["B4"], N * r).reshape(N, r)))
        return self.chain(out, q0, s0)

    # ---- Mamba-2 decode step around the linears ----------------------------
    def add_rmsnorm_quant(self, u, w, eps, delta=None):
        """Returns (u_out, o, Q, s): u_out = u + delta, o = rmsnorm(u_out) * w
        (fp32), (Q, s) = quantise(o)."""
        u = np.ascontiguousarray(u, np.float32)
        w = np.ascontiguousarray(w, np.float32)
        M, d = u.shape
        dl = None if delta is None else np.ascontiguousarray(delta, np.float32)
        u_out = np.zeros((M, d), np.float32)
        o = np.zeros((M, d), np.float32)
        q = np.zeros((M, d), np.int8)
        s = np.zeros((M,), np.float32)
        st = self.lib.dfssm_ref_add_rmsnorm_quant(_p(u), _p(dl), _p(w), float(eps), M, d, _p(u_out), _p(o),
                                                 _p(q), _p(s))
        if st != OK:
            raise OracleError(st)
        return u_out, o, q, s

    def ssm_step(self, zxbcdt, conv_state, ssm_state, conv_w, conv_b, dt_bias, A_log, D, d_inner, d_state,
                 headdim):
        """One token per sequence through the conv step and the SSM step.
        conv_state [M, conv_dim, 4] (position 3 newest) and ssm_state
        [M, H, P, N] are copied, not modified.  Returns (y [M, d_inner],
        xbc [M, conv_dim], conv_state', ssm_state')."""
        zx = np.ascontiguousarray(zxbcdt, np.float32)
        M, ld = zx.shape
        conv_dim = d_inner + 2 * d_state
        cs = np.array(conv_state, np.float32, copy=True, order="C")
        hs = np.array(ssm_state, np.float32, copy=True, order="C")
        if cs.shape != (M, conv_dim, 4) or hs.shape != (M, d_inner // headdim, headdim, d_state):
            raise ValueError("state shapes")
        arrs = [np.ascontiguousarray(a, np.float32) for a in (conv_w, conv_b, dt_bias, A_log, D)]
        y = np.zeros((M, d_inner), np.float32)
        xbc = np.zeros((M, conv_dim), np.float32)
        st = self.lib.dfssm_ref_ssm_step(_p(zx), ld, M, d_inner, d_state, headdim, _p(cs), *[_p(a) for a in arrs],
                                         _p(hs), _p(y), _p(xbc))
        if st != OK:
            raise OracleError(st)
        return y, xbc, cs, hs

    def gate_norm_quant(self, y, z, w, eps):
        """Returns (o, Q, s): o = rmsnorm(y * silu(z)) * w, (Q, s) = quantise(o)."""
        y = np.ascontiguousarray(y, np.float32)
        z = np.ascontiguousarray(z, np.float32)
        w = np.ascontiguousarray(w, np.float32)
        M, d = y.shape
        o = np.zeros((M, d), np.float32)
        q = np.zeros((M, d), np.int8)
        s = np.zeros((M,), np.float32)
        st = self.lib.dfssm_ref_gate_norm_quant(_p(y), _p(z), z.shape[1], _p(w), float(eps), M, d, _p(o), _p(q),
                                               _p(s))
        if st != OK:
            raise OracleError(st)
        return o, q, s

    def threads(self) -> int:
        return self.lib.dfssm_ref_threads()

    def set_threads(self, n: int) -> None:
        """Thread count of later oracle calls (timing only; results do not depend on it)."""
        self.lib.dfssm_ref_set_threads(int(n))


class OracleError(RuntimeError):
    def __init__(self, status: int):
        super().__init__(f"oracle status {status}")
        self.status = status


_default: Optional[Oracle] = None


def get() -> Oracle:
    """The oracle built from dfssm_ref.c (built on first use)."""
    global _default
    if _default is None:
        _default = Oracle(LIB)
    return _default
