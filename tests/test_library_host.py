"""Host-side checks of the HIP library (no GPU needed): it loads, exports
every function include/dfssm.h declares, and rejects invalid arguments on the
host before any HIP call.  Also checks the product/oracle separation."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dfssm.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dfssm_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def dl():
    import paper_2606_10932_amd as D
    return D


def test_exports_every_declared_function(dl):
    names = header_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(dl.lib, n), n          # dlsym succeeds
    assert set(names) == set(dl.EXPORTS)


def test_version_and_status_strings(dl):
    assert dl.lib.dfssm_version().decode().startswith("dfssm")
    for st in range(7):
        assert dl.lib.dfssm_status_string(st).decode() not in ("", "unknown status")
    assert dl.lib.dfssm_status_string(99).decode() == "unknown status"


def _lin(dl, M=1, K=64, N=8, r=4, q=16, s=16, w=16, al=16, A=16, B=16, be=16, y=16, ws=16,
         wsb=1 << 20, path=0):
    return dl.lib.dfssm_scaffold_lora_linear_ex(q, s, M, K, N, r, w, al, A, B, be, y, path, None, None,
                                                None, ws, wsb, None)


def test_linear_validation(dl):
    # fake, aligned, non-null "device" pointers: every call below must be
    # rejected on the host before anything touches a device
    assert _lin(dl, K=48) == dl.ERR_SHAPE
    assert _lin(dl, K=0) == dl.ERR_SHAPE
    assert _lin(dl, K=65536 + 32) == dl.ERR_SHAPE
    assert _lin(dl, M=-1) == dl.ERR_SHAPE
    assert _lin(dl, N=-1) == dl.ERR_SHAPE
    assert _lin(dl, r=257) == dl.ERR_SHAPE
    assert _lin(dl, r=-1) == dl.ERR_SHAPE
    assert _lin(dl, path=7) == dl.ERR_SHAPE
    assert _lin(dl, q=None) == dl.ERR_NULL
    assert _lin(dl, w=None) == dl.ERR_NULL
    assert _lin(dl, ws=None) == dl.ERR_NULL
    assert _lin(dl, A=None) == dl.ERR_NULL           # r > 0 needs A, B, beta
    assert _lin(dl, be=None) == dl.ERR_NULL
    assert _lin(dl, q=17) == dl.ERR_ALIGN
    assert _lin(dl, y=20) == dl.ERR_ALIGN
    assert _lin(dl, wsb=10) == dl.ERR_WORKSPACE
    assert "workspace" in dl.last_error()
    # empty problems are accepted as no-ops
    assert _lin(dl, M=0, q=None, s=None) == dl.OK
    assert _lin(dl, N=0, w=None) == dl.OK
    # the plain entry point needs y
    assert dl.lib.dfssm_scaffold_lora_linear(16, 16, 1, 64, 8, 0, 16, 16, None, None, None, None, 16,
                                              1 << 20, None) == dl.ERR_NULL


def test_quantize_validation(dl):
    f = dl.lib.dfssm_quantize_act
    assert f(16, 2, 1, 64, 64, 16, 16, None) == dl.ERR_SHAPE      # dtype
    assert f(16, dl.F16, 1, 48, 64, 16, 16, None) == dl.ERR_SHAPE
    assert f(16, dl.F16, 1, 64, 32, 16, 16, None) == dl.ERR_SHAPE  # ldx < K
    assert f(None, dl.F16, 1, 64, 64, 16, 16, None) == dl.ERR_NULL
    assert f(17, dl.F16, 1, 64, 64, 16, 16, None) == dl.ERR_ALIGN  # fp16 needs 2-byte alignment
    assert f(18, dl.F32, 1, 64, 64, 16, 16, None) == dl.ERR_ALIGN
    assert f(16, dl.F16, 1, 64, 64, 24, 16, None) == dl.ERR_ALIGN
    assert f(None, dl.F16, 0, 64, 64, None, None, None) == dl.OK   # M = 0


def test_chain_validation(dl):
    L = dl.Layer
    good = dict(w_bits=16, alpha=16, A=16, B=16, beta=16, K=64, N=96, r=4)
    arr = (L * 2)(L(**good), L(**dict(good, K=128)))              # K_1 = 128 > N_0 = 96
    f = dl.lib.dfssm_scaffold_lora_chain
    assert f(arr, 2, 1, 16, 16, 16, 16, 1 << 30, None) == dl.ERR_SHAPE
    arr = (L * 2)(L(**good), L(**dict(good, K=64)))
    assert f(arr, 2, 5, 16, 16, 16, 16, 1 << 30, None) == dl.ERR_UNSUPPORTED   # M > 4
    assert f(arr, 2, 1, 16, 16, 16, 16, 8, None) == dl.ERR_WORKSPACE
    assert f(arr, 2, 1, None, 16, 16, 16, 1 << 30, None) == dl.ERR_NULL
    arr = (L * 1)(L(**dict(good, A=None)))
    assert f(arr, 1, 1, 16, 16, 16, 16, 1 << 30, None) == dl.ERR_NULL
    assert "layer 0" in dl.last_error()
    assert f(arr, 0, 1, None, None, None, None, 0, None) == dl.OK
    assert dl.lib.dfssm_chain_workspace_bytes(arr, 1, 1) > 0
    # prepare / run / status validate the same way, before any HIP call
    arr = (L * 2)(L(**good), L(**dict(good, K=128)))
    assert dl.lib.dfssm_chain_prepare(arr, 2, 1, 16, 1 << 30, None) == dl.ERR_SHAPE
    assert dl.lib.dfssm_chain_run(arr, 2, 1, 16, 16, 16, 16, 1 << 30, None) == dl.ERR_SHAPE
    arr = (L * 2)(L(**good), L(**dict(good, K=64)))
    assert dl.lib.dfssm_chain_prepare(arr, 2, 1, 16, 8, None) == dl.ERR_WORKSPACE
    assert dl.lib.dfssm_chain_run(arr, 2, 1, None, 16, 16, 16, 1 << 30, None) == dl.ERR_NULL
    st = ctypes.c_uint(7)
    assert dl.lib.dfssm_chain_status(arr, 2, 1, 16, 8, ctypes.byref(st), None) == dl.ERR_WORKSPACE
    assert dl.lib.dfssm_chain_status(arr, 2, 1, 16, 1 << 30, None, None) == dl.ERR_NULL
    # the read-floor diagnostic validates before any HIP call
    pp, ppb = dl.lib.dfssm_exchange_pingpong, dl.lib.dfssm_exchange_pingpong_bytes()
    ns = ctypes.c_double(1.0)
    assert ppb >= 256 * 64 * 8
    assert pp(0, 10, 0, 16, ppb, ctypes.byref(ns), None) == dl.ERR_SHAPE and ns.value == 0.0
    assert pp(129, 10, 0, 16, ppb, ctypes.byref(ns), None) == dl.ERR_SHAPE
    assert pp(1, 0, 0, 16, ppb, ctypes.byref(ns), None) == dl.ERR_SHAPE
    assert pp(1, 10, 0, None, ppb, ctypes.byref(ns), None) == dl.ERR_NULL
    assert pp(1, 10, 0, 16, ppb - 1, ctypes.byref(ns), None) == dl.ERR_WORKSPACE
    assert pp(1, 10, 0, 16, ppb, None, None) == dl.ERR_NULL
    rf = dl.lib.dfssm_read_floor
    assert dl.lib.dfssm_read_floor_sink_words(2923008) == 4 * 357   # one word per wave
    assert dl.lib.dfssm_read_floor_sink_words(0) == 4
    assert rf(16, 17, 16, 4, None) == dl.ERR_SHAPE         # not a multiple of 16
    assert rf(16, 32, None, 4, None) == dl.ERR_NULL        # no sink
    assert rf(16, 32, 18, 4, None) == dl.ERR_ALIGN         # sink not 4-byte aligned
    assert rf(16, 16 * 513, 16, 4, None) == dl.ERR_WORKSPACE   # two blocks: 8 words
    assert rf(None, 32, 16, 4, None) == dl.ERR_NULL
    assert rf(24, 32, 16, 4, None) == dl.ERR_ALIGN
    # the loads-only diagnostic: same validation; chains the persistent kernel
    # does not take (K = 64 here) are refused before any HIP call
    fs = dl.lib.dfssm_chain_stream_floor
    assert fs(arr, 2, None, 1 << 30, None) == dl.ERR_NULL
    assert fs(arr, 2, 16, 8, None) == dl.ERR_WORKSPACE
    assert fs(arr, 2, 16, 1 << 30, None) == dl.ERR_UNSUPPORTED
    arr = (L * 2)(L(**good), L(**dict(good, K=128)))
    assert fs(arr, 2, 16, 1 << 30, None) == dl.ERR_SHAPE


def test_make_layers_keeps_tensors(dl):
    """The layer array holds its tensors: dropping the caller's list must not
    free memory the array still points at."""
    import gc
    import weakref
    import torch
    refs = []

    def build():
        ly = [dict(w_bits=torch.zeros((96, 2), dtype=torch.int32), alpha=torch.zeros(96),
                   A=torch.zeros((4, 64), dtype=torch.int8), B=torch.zeros((96, 4), dtype=torch.int8),
                   beta=torch.zeros(96))]
        refs.append(weakref.ref(ly[0]["w_bits"]))
        return dl.make_layers(ly)
    arr = build()
    gc.collect()
    assert refs[0]() is not None and refs[0]().data_ptr() == arr[0].w_bits
    del arr
    gc.collect()
    assert refs[0]() is None


def test_embedding_validation(dl):
    g = dl.lib.dfssm_embed_gather      # E, scale, V, d, tok, M, x, stream
    assert g(16, 16, 100, 24, 16, 1, 16, None) == dl.ERR_SHAPE       # d % 16
    assert g(16, 16, 100, 0, 16, 1, 16, None) == dl.ERR_SHAPE
    assert g(16, 16, 0, 64, 16, 1, 16, None) == dl.ERR_SHAPE         # empty table
    assert g(16, 16, 100, 64, 16, -1, 16, None) == dl.ERR_SHAPE
    assert g(None, 16, 100, 64, 16, 1, 16, None) == dl.ERR_NULL
    assert g(16, 16, 100, 64, None, 1, 16, None) == dl.ERR_NULL
    assert g(16, 16, 100, 64, 16, 1, 20, None) == dl.ERR_ALIGN
    assert g(None, None, 100, 64, None, 0, None, None) == dl.OK      # M = 0
    h = dl.lib.dfssm_lm_head           # q, s, M, d, E, scale, V, logits, acc, stream
    assert h(16, 16, 1, 24, 16, 16, 100, 16, None, None) == dl.ERR_SHAPE
    assert h(16, 16, 1, 16384 + 16, 16, 16, 100, 16, None, None) == dl.ERR_SHAPE
    assert h(16, 16, 1, 64, 16, 16, -1, 16, None, None) == dl.ERR_SHAPE
    assert h(16, 16, -1, 64, 16, 16, 100, 16, None, None) == dl.ERR_SHAPE
    assert h(16, 16, 1, 64, 16, 16, 100, None, None, None) == dl.ERR_NULL   # no output
    assert h(16, 16, 1, 64, None, 16, 100, 16, None, None) == dl.ERR_NULL
    assert h(16, 16, 1, 64, 16, 16, 100, 16, 36, None) == dl.ERR_ALIGN
    assert h(None, None, 0, 64, None, None, 100, None, None, None) == dl.OK
    assert h(None, None, 1, 64, None, None, 0, None, None, None) == dl.OK   # V = 0


def test_mamba_step_validation(dl):
    n = dl.lib.dfssm_add_rmsnorm_quant   # u, delta, w, eps, M, d, u_out, q, s, stream
    assert n(16, None, 16, 1e-5, 1, 30, None, 16, 16, None) == dl.ERR_SHAPE      # d % 4
    assert n(16, None, 16, 1e-5, 1, 16384 + 4, None, 16, 16, None) == dl.ERR_SHAPE
    assert n(16, None, 16, -1.0, 1, 64, None, 16, 16, None) == dl.ERR_SHAPE      # eps < 0
    assert n(16, None, 16, float("nan"), 1, 64, None, 16, 16, None) == dl.ERR_SHAPE
    assert n(None, None, 16, 1e-5, 1, 64, None, 16, 16, None) == dl.ERR_NULL
    assert n(16, 20, 16, 1e-5, 1, 64, None, 16, 16, None) == dl.ERR_ALIGN        # delta
    assert n(None, None, None, 1e-5, 0, 64, None, None, None, None) == dl.OK     # M = 0
    g = dl.lib.dfssm_gate_norm_quant     # y, z, ldz, w, eps, M, d, q, s, stream
    assert g(16, 16, 32, 16, 1e-5, 1, 64, 16, 16, None) == dl.ERR_SHAPE           # ldz < d
    assert g(16, 16, 66, 16, 1e-5, 1, 64, 16, 16, None) == dl.ERR_SHAPE           # ldz % 4
    assert g(16, None, 64, 16, 1e-5, 1, 64, 16, 16, None) == dl.ERR_NULL
    f = dl.lib.dfssm_ssm_step

    def ssm(ld=8512, M=1, di=4096, N=128, P=64, step=0, zx=16, xbc=None):
        return f(zx, ld, M, di, N, P, step, 16, 16, 16, 16, 16, 16, 16, 16, xbc, None)
    assert ssm(P=32) == dl.ERR_UNSUPPORTED
    assert ssm(N=96) == dl.ERR_UNSUPPORTED
    assert ssm(di=4000) == dl.ERR_SHAPE
    assert ssm(ld=8511) == dl.ERR_SHAPE
    assert ssm(step=-1) == dl.ERR_SHAPE
    assert ssm(M=-1) == dl.ERR_SHAPE
    assert ssm(zx=None) == dl.ERR_NULL
    assert ssm(xbc=24) == dl.ERR_ALIGN
    assert ssm(M=0, zx=None) == dl.OK


def test_model_step_validation(dl):
    import ctypes
    good_in = dl.Layer(16, 16, 16, 16, 16, 2048, 8512, 64)
    good_out = dl.Layer(16, 16, 16, 16, 16, 4096, 2048, 64)
    lay = (dl.Mamba2Layer * 2)(dl.Mamba2Layer(16, good_in, 16, 16, 16, 16, 16, 16, good_out),
                               dl.Mamba2Layer(16, good_in, 16, 16, 16, 16, 16, 16, good_out))

    def model(**kw):
        f = dict(d_model=2048, d_state=128, n_layers=2, vocab=50280, eps=1e-5, E=16, E_scale=16, norm_f=16)
        f.update(kw)
        return dl.Mamba2Model(f["d_model"], f["d_state"], f["n_layers"], f["vocab"], f["eps"], f["E"],
                              f["E_scale"], f["norm_f"], lay)

    step = dl.lib.dfssm_mamba2_decode_step    # model, M, tok, step, ring, state, logits, ws, bytes, stream

    def run(m, M=1, ws_bytes=1 << 40, tok=16, t=0):
        return step(ctypes.byref(m), M, tok, t, 16, 16, 16, 16, ws_bytes, None)
    assert run(model(d_model=2000)) == dl.ERR_SHAPE
    assert run(model(d_model=2080)) == dl.ERR_SHAPE          # not a multiple of 128
    assert run(model(d_state=96)) == dl.ERR_UNSUPPORTED
    assert run(model(vocab=0)) == dl.ERR_SHAPE
    assert run(model(), M=0) == dl.ERR_SHAPE
    assert run(model(), t=-1) == dl.ERR_SHAPE
    assert run(model(E=None)) == dl.ERR_NULL
    assert run(model(), tok=None) == dl.ERR_NULL
    assert run(model(), ws_bytes=64) == dl.ERR_WORKSPACE
    lay[1].out_proj.N = 2047
    assert run(model()) == dl.ERR_SHAPE and "layer 1" in dl.last_error()
    lay[1].out_proj.N = 2048
    lay[0].conv_b = None
    assert run(model()) == dl.ERR_NULL and "layer 0" in dl.last_error()
    lay[0].conv_b = 16
    m = model()
    c, s = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert dl.lib.dfssm_mamba2_state_bytes(ctypes.byref(m), 3, ctypes.byref(c), ctypes.byref(s)) == dl.OK
    assert c.value == 2 * 3 * 4 * 4352 * 4 and s.value == 2 * 3 * 64 * 64 * 128 * 4
    assert dl.lib.dfssm_mamba2_workspace_bytes(ctypes.byref(m), 1) > 0
    # int4 factors: lora_bits 4 (0 and 8 mean int8), even ranks, and room
    # for the factors the prefill path expands
    w8 = dl.lib.dfssm_mamba2_workspace_bytes(ctypes.byref(m), 1024)
    lay[1].lora_bits = 5
    assert run(model()) == dl.ERR_SHAPE and "layer 1" in dl.last_error() and "lora_bits" in dl.last_error()
    lay[0].lora_bits = lay[1].lora_bits = 4
    lay[0].in_proj.r = 63
    assert run(model()) == dl.ERR_SHAPE and "even" in dl.last_error()
    lay[0].in_proj.r = 64
    w4 = dl.lib.dfssm_mamba2_workspace_bytes(ctypes.byref(m), 1024)
    assert w4 >= w8 + 64 * 4096 + 2048 * 64     # out_proj: the larger linear workspace
    assert dl.lib.dfssm_mamba2_workspace_bytes(ctypes.byref(m), 1) > 0
    # the fused step's region: at M = 1 only, for the 1.3B layer shape with
    # int8 factors (r % 4 == 0) or int4 ones (r % 8 == 0); not for int4 at r = 12
    lay[0].lora_bits = lay[1].lora_bits = 4
    w1_i4 = dl.lib.dfssm_mamba2_workspace_bytes(ctypes.byref(m), 1)
    lay[0].in_proj.r = lay[0].out_proj.r = lay[1].in_proj.r = lay[1].out_proj.r = 12
    w1_i4_r12 = dl.lib.dfssm_mamba2_workspace_bytes(ctypes.byref(m), 1)
    lay[0].lora_bits = lay[1].lora_bits = 8
    w1_r12 = dl.lib.dfssm_mamba2_workspace_bytes(ctypes.byref(m), 1)
    lay[0].in_proj.r = lay[0].out_proj.r = lay[1].in_proj.r = lay[1].out_proj.r = 64
    w1 = dl.lib.dfssm_mamba2_workspace_bytes(ctypes.byref(m), 1)
    assert w1_r12 > w1_i4_r12 + 800 * 1024   # 2 layers: ~0.9 MB of fused region, int8 only at r = 12
    assert w1_i4 > w1_i4_r12 + 800 * 1024 and w1 > 800 * 1024
    # prepare / release / status validate on the host
    prep, stat = dl.lib.dfssm_mamba2_prepare, dl.lib.dfssm_mamba2_status
    assert prep(None, 1, 16, 1 << 40, None) == dl.ERR_NULL
    assert prep(ctypes.byref(model(d_state=96)), 1, 16, 1 << 40, None) == dl.ERR_UNSUPPORTED
    assert prep(ctypes.byref(m), 1, None, 1 << 40, None) == dl.ERR_NULL
    assert prep(ctypes.byref(m), 1, 16, 64, None) == dl.ERR_WORKSPACE
    assert dl.lib.dfssm_mamba2_release(None) == dl.OK and dl.lib.dfssm_mamba2_release(16) == dl.OK
    st = ctypes.c_uint(7)
    assert stat(ctypes.byref(m), 1, 16, 1 << 40, None, None) == dl.ERR_NULL
    assert stat(ctypes.byref(m), 1, 16, 64, ctypes.byref(st), None) == dl.ERR_WORKSPACE
    # an unprepared workspace: no device read, status 0
    assert stat(ctypes.byref(m), 1, 16, 1 << 40, ctypes.byref(st), None) == dl.OK and st.value == 0
    # the path query: the per-kernel sequence on an unprepared workspace
    fp, fz = dl.lib.dfssm_mamba2_fused_path, ctypes.c_int(7)
    assert fp(ctypes.byref(m), 1, 16, 1 << 40, None) == dl.ERR_NULL
    assert fp(ctypes.byref(m), 1, 16, 64, ctypes.byref(fz)) == dl.ERR_WORKSPACE
    assert fp(ctypes.byref(m), 1, 16, 1 << 40, ctypes.byref(fz)) == dl.OK and fz.value == 0


def test_int4_linear_validation(dl):
    f = dl.lib.dfssm_scaffold_lora_linear_i4   # q, s, M, K, N, r, w, alpha, A4, B4, beta, y, path, acc*3, ws, bytes, stream

    def lin(M=1, K=64, N=8, r=4, A4=16, path=0, wsb=1 << 20, y=16):
        return f(16, 16, M, K, N, r, 16, 16, A4, 16, 16, y, path, None, None, None, 16, wsb, None)
    assert lin(r=5) == dl.ERR_SHAPE                 # odd rank: half a byte
    assert lin(K=48) == dl.ERR_SHAPE
    assert lin(A4=None) == dl.ERR_NULL
    assert lin(A4=24) == dl.ERR_ALIGN
    assert lin(path=9) == dl.ERR_SHAPE
    assert lin(M=513, path=3) == dl.ERR_UNSUPPORTED
    need = dl.lib.dfssm_linear_i4_workspace_bytes(1, 64, 8, 4)
    assert need > dl.linear_workspace_bytes(1, 64, 8, 4)
    assert lin(wsb=need - 1) == dl.ERR_WORKSPACE
    assert lin(M=0) == dl.OK


def test_workspace_sizes(dl):
    a = dl.linear_workspace_bytes(1, 2048, 8512, 64)
    b = dl.linear_workspace_bytes(2048, 2048, 8512, 64)
    assert 0 < a < b
    assert dl.linear_workspace_bytes(1, 2048, 8512, 0) > 0


def _imports(path):
    out = []
    for dirpath, _, files in os.walk(path):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".hpp", ".h", ".c")):
                out.append((os.path.join(dirpath, f), open(os.path.join(dirpath, f)).read()))
    return out


def test_product_and_oracle_are_separate():
    for p, text in _imports(os.path.join(ROOT, "paper_2606_10932_amd")):
        assert not re.search(r"^\s*(from|import)\s+oracle\b", text, re.M), p
        assert "dfssm_ref" not in text, p
    for p, text in _imports(os.path.join(ROOT, "oracle")):
        assert "paper_2606_10932_amd" not in text, p
        assert not re.search(r'#\s*include\s*[<"](dfssm\.h|dfssm_internal)', text), p
    for p, text in _imports(os.path.join(ROOT, "dfssm_synth")):
        assert "oracle" not in text.replace("imports neither the oracle", ""), p
        assert "paper_2606_10932_amd" not in text, p
