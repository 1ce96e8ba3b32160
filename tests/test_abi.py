"""C-ABI library: loads, exports every declared symbol, rejects bad arguments
before touching the GPU (CPU only; no compute calls)."""

import ctypes
import os

import pytest
import torch

from paper_2609_08368_amd import rl_attn as ra

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x100000          # never dereferenced: every call below fails host validation first


def fake(shape, dtype, ptr=FAKE, strides=None):
    v = ra.RlTensor()
    v.data = ptr
    v.dtype = dtype
    v.ndim = len(shape)
    st = strides
    if st is None:
        st, acc = [], 1
        for s in reversed(shape):
            st.insert(0, acc)
            acc *= s
    for i, s in enumerate(shape):
        v.shape[i] = s
        v.strides[i] = st[i]
    return v


def decode_args(B=2, Hq=8, Hkv=2, P=16, npages=10, maxp=4, D=128):
    return dict(
        q=fake([B, Hq, D], ra.RL_BF16), k=fake([npages, P, Hkv, D], ra.RL_BF16),
        v=fake([npages, P, Hkv, D], ra.RL_BF16), bt=fake([B, maxp], ra.RL_I32),
        lens=fake([B], ra.RL_I32), out=fake([B, Hq, D], ra.RL_BF16), lse=None, opts=None)


def call_decode(a):
    r = ctypes.byref
    return ra.lib().rl_attn_decode_ex(r(a["q"]), r(a["k"]), r(a["v"]), r(a["bt"]), r(a["lens"]),
                                      ctypes.c_float(0.088), r(a["out"]),
                                      r(a["lse"]) if a["lse"] is not None else None,
                                      r(a["opts"]) if a["opts"] is not None else None, None)


def test_library_exports_every_declared_symbol():
    names = ra.header_functions()
    assert {"rl_attn_decode", "rl_attn_extend", "rl_attn_merge", "rl_attn_last_error"} <= set(names)
    lib = ra.lib()
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("mutate,code,needle", [
    (lambda a: a.update(q=None) or a, "RL_ERR_INVALID_ARG", "q is NULL"),
    (lambda a: setattr(a["q"], "dtype", ra.RL_F32) or a, "RL_ERR_DTYPE", "q must be bf16"),
    (lambda a: a.update(q=fake([2, 8], ra.RL_BF16)) or a, "RL_ERR_SHAPE", "q must have 3"),
    (lambda a: a.update(**decode_args(D=64)) or a, "RL_ERR_UNSUPPORTED", "head dimension must be 128"),
    (lambda a: a.update(**decode_args(P=48)) or a, "RL_ERR_UNSUPPORTED", "page size"),
    (lambda a: a.update(**decode_args(P=256)) or a, "RL_ERR_UNSUPPORTED", "page size"),
    (lambda a: a.update(**decode_args(P=4)) or a, "RL_ERR_UNSUPPORTED", "page size"),
    (lambda a: a.update(**decode_args(Hq=6, Hkv=4)) or a, "RL_ERR_SHAPE", "multiple of KV heads"),
    (lambda a: a.update(bt=fake([3, 4], ra.RL_I32)) or a, "RL_ERR_SHAPE", "block_table.shape[0]"),
    (lambda a: a.update(bt=fake([2, 4], ra.RL_F32)) or a, "RL_ERR_DTYPE", "block_table must be int32"),
    (lambda a: a.update(lens=fake([3], ra.RL_I32)) or a, "RL_ERR_SHAPE", "seq_lens.shape[0]"),
    (lambda a: a.update(lens=fake([2], ra.RL_F32)) or a, "RL_ERR_DTYPE", "seq_lens must be int32"),
    (lambda a: a.update(out=fake([2, 8, 128], ra.RL_I32)) or a, "RL_ERR_DTYPE", "out must be bf16 or f32"),
    (lambda a: a.update(out=fake([2, 4, 128], ra.RL_BF16)) or a, "RL_ERR_SHAPE", "out shape"),
    (lambda a: a.update(lse=fake([2, 7], ra.RL_F32)) or a, "RL_ERR_SHAPE", "lse_out shape"),
    (lambda a: a.update(lse=fake([2, 8], ra.RL_BF16)) or a, "RL_ERR_DTYPE", "lse_out must be f32"),
    (lambda a: a.update(k=fake([10, 16, 2, 128], ra.RL_BF16, strides=[4096, 256, 128, 2])) or a,
     "RL_ERR_UNSUPPORTED", "last stride"),
    (lambda a: a.update(q=fake([2, 8, 128], ra.RL_BF16, ptr=FAKE + 2)) or a, "RL_ERR_UNSUPPORTED", "aligned"),
    (lambda a: a.update(v=fake([10, 16, 2, 128], ra.RL_BF16, ptr=0)) or a, "RL_ERR_INVALID_ARG", "v_pages.data"),
    (lambda a: a.update(v=fake([11, 16, 2, 128], ra.RL_BF16)) or a, "RL_ERR_SHAPE", "shapes differ"),
    # multi-token decode: q [B, n, Hq, 128] with 1 <= n <= 64, out and lse [B, n, Hq] to match
    (lambda a: a.update(q=fake([2, 65, 8, 128], ra.RL_BF16), out=fake([2, 65, 8, 128], ra.RL_BF16)) or a,
     "RL_ERR_UNSUPPORTED", "query tokens per sequence"),
    (lambda a: a.update(q=fake([2, 0, 8, 128], ra.RL_BF16), out=fake([2, 0, 8, 128], ra.RL_BF16)) or a,
     "RL_ERR_UNSUPPORTED", "query tokens per sequence"),
    (lambda a: a.update(q=fake([2, 4, 8, 128], ra.RL_BF16)) or a, "RL_ERR_SHAPE", "out must have 4"),
    (lambda a: a.update(q=fake([2, 4, 8, 128], ra.RL_BF16), out=fake([2, 4, 8, 128], ra.RL_BF16),
                        lse=fake([2, 8], ra.RL_F32)) or a, "RL_ERR_SHAPE", "lse_out must have 3"),
    (lambda a: a.update(q=fake([2, 4, 8, 128], ra.RL_BF16), out=fake([2, 4, 8, 128], ra.RL_BF16),
                        lse=fake([2, 3, 8], ra.RL_F32)) or a, "RL_ERR_SHAPE", "lse_out shape"),
    # (sequence, query row) pairs must fit 32-bit indices
    (lambda a: a.update(**decode_args(B=1 << 22, Hq=1024, Hkv=8)) or a, "RL_ERR_UNSUPPORTED", "too large"),
])
def test_decode_validation(mutate, code, needle):
    a = mutate(decode_args())
    if a["q"] is None:
        rc = ra.lib().rl_attn_decode_ex(None, ctypes.byref(a["k"]), ctypes.byref(a["v"]), ctypes.byref(a["bt"]),
                                        ctypes.byref(a["lens"]), ctypes.c_float(1.0), ctypes.byref(a["out"]),
                                        None, None, None)
    else:
        rc = call_decode(a)
    assert ra.STATUS[rc] == code, ra.last_error()
    assert needle in ra.last_error()


@pytest.mark.parametrize("field,value,needle", [
    ("split_tokens", 100, "split_tokens"), ("split_tokens", -64, "split_tokens"),
    ("prefix_share", 7, "prefix_share"), ("validate", 2, "validate"), ("deterministic", -1, "deterministic")])
def test_option_validation(field, value, needle):
    a = decode_args()
    o = ra.RlOpts()
    setattr(o, field, value)
    a["opts"] = o
    assert ra.STATUS[call_decode(a)] == "RL_ERR_INVALID_ARG"
    assert needle in ra.last_error()
    o2 = ra.RlOpts()
    o2.reserved[3] = 1
    a["opts"] = o2
    assert ra.STATUS[call_decode(a)] == "RL_ERR_INVALID_ARG" and "reserved" in ra.last_error()


def test_empty_batch_is_a_no_op():
    a = decode_args(B=0)
    assert call_decode(a) == 0


def test_extend_validation():
    r = ctypes.byref
    B = 3
    q = fake([10, 8, 128], ra.RL_BF16)
    k = fake([20, 16, 2, 128], ra.RL_BF16)
    bt = fake([B, 4], ra.RL_I32)
    kv = fake([B], ra.RL_I32)
    out = fake([10, 8, 128], ra.RL_BF16)
    bad_indptr = fake([B], ra.RL_I32)
    rc = ra.lib().rl_attn_extend(r(q), r(bad_indptr), r(k), r(k), r(bt), r(kv), ctypes.c_float(1.0), r(out), None)
    assert ra.STATUS[rc] == "RL_ERR_SHAPE" and "qo_indptr" in ra.last_error()
    indptr = fake([B + 1], ra.RL_F32)
    rc = ra.lib().rl_attn_extend(r(q), r(indptr), r(k), r(k), r(bt), r(kv), ctypes.c_float(1.0), r(out), None)
    assert ra.STATUS[rc] == "RL_ERR_DTYPE"
    indptr = fake([B + 1], ra.RL_I32)
    out_bad = fake([9, 8, 128], ra.RL_BF16)
    rc = ra.lib().rl_attn_extend(r(q), r(indptr), r(k), r(k), r(bt), r(kv), ctypes.c_float(1.0), r(out_bad), None)
    assert ra.STATUS[rc] == "RL_ERR_SHAPE"
    q0 = fake([0, 8, 128], ra.RL_BF16)
    out0 = fake([0, 8, 128], ra.RL_BF16)
    rc = ra.lib().rl_attn_extend(r(q0), r(indptr), r(k), r(k), r(bt), r(kv), ctypes.c_float(1.0), r(out0), None)
    assert rc == 0, ra.last_error()


def test_merge_validation():
    r = ctypes.byref
    o = fake([4, 3, 8, 128], ra.RL_F32)
    l = fake([4, 3, 8], ra.RL_F32)
    n = fake([4], ra.RL_I32)
    out = fake([4, 8, 128], ra.RL_F32)
    assert ra.STATUS[ra.lib().rl_attn_merge(r(o), r(fake([4, 2, 8], ra.RL_F32)), r(n), r(out), None, None)] == "RL_ERR_SHAPE"
    assert ra.STATUS[ra.lib().rl_attn_merge(r(o), r(l), r(fake([4], ra.RL_F32)), r(out), None, None)] == "RL_ERR_DTYPE"
    assert ra.STATUS[ra.lib().rl_attn_merge(r(fake([4, 3, 8, 64], ra.RL_F32)), r(l), r(n), r(fake([4, 8, 64], ra.RL_F32)), None, None)] == "RL_ERR_UNSUPPORTED"


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-GPU error path")
def test_valid_call_without_gpu_reports_hip_error():
    rc = call_decode(decode_args())
    assert ra.STATUS[rc] in ("RL_ERR_HIP", "RL_ERR_WORKSPACE"), ra.last_error()


@pytest.mark.parametrize("scale", [float("nan"), 0.0, -0.1, float("inf")])
def test_scale_must_be_positive_and_finite(scale):
    a = decode_args()
    r = ctypes.byref
    rc = ra.lib().rl_attn_decode_ex(r(a["q"]), r(a["k"]), r(a["v"]), r(a["bt"]), r(a["lens"]), ctypes.c_float(scale),
                                    r(a["out"]), None, None, None)
    assert ra.STATUS[rc] == "RL_ERR_INVALID_ARG" and "scale" in ra.last_error()


def test_diagnostics_validate_arguments():
    lib, d = ra.lib(), ctypes.c_double()
    r = ctypes.byref
    assert ra.STATUS[lib.rl_attn_diag_read_bandwidth(None, 1024, 1, r(d), None)] == "RL_ERR_INVALID_ARG"
    assert ra.STATUS[lib.rl_attn_diag_read_bandwidth(ctypes.c_void_p(FAKE), 1000, 1, r(d), None)] == "RL_ERR_INVALID_ARG"
    assert ra.STATUS[lib.rl_attn_diag_read_bandwidth(ctypes.c_void_p(FAKE + 4), 1024, 1, r(d), None)] == "RL_ERR_INVALID_ARG"
    assert ra.STATUS[lib.rl_attn_diag_read_bandwidth(ctypes.c_void_p(FAKE), 1024, 0, r(d), None)] == "RL_ERR_INVALID_ARG"
    assert ra.STATUS[lib.rl_attn_diag_mfma_bf16(0, r(d), None)] == "RL_ERR_INVALID_ARG"
    assert ra.STATUS[lib.rl_attn_diag_mfma_bf16((1 << 24) + 1, r(d), None)] == "RL_ERR_INVALID_ARG"
    assert ra.STATUS[lib.rl_attn_diag_mfma_bf16(10, None, None)] == "RL_ERR_INVALID_ARG"


def fp8_decode_args(Hkv=2):
    a = decode_args(Hkv=Hkv)
    a["k"] = fake([10, 16, Hkv, 128], ra.RL_FP8_E4M3)
    a["v"] = fake([10, 16, Hkv, 128], ra.RL_FP8_E4M3)
    a["ks"] = fake([Hkv], ra.RL_F32)
    a["vs"] = fake([Hkv], ra.RL_F32)
    return a


def call_decode_fp8(a):
    r = ctypes.byref
    opt = lambda x: r(x) if x is not None else None
    return ra.lib().rl_attn_decode_fp8(r(a["q"]), r(a["k"]), r(a["v"]), opt(a["ks"]), opt(a["vs"]), r(a["bt"]),
                                       r(a["lens"]), ctypes.c_float(0.088), r(a["out"]), None, None, None)


@pytest.mark.parametrize("mutate,code,needle", [
    (lambda a: a.update(k=fake([10, 16, 2, 128], ra.RL_BF16)) or a, "RL_ERR_DTYPE", "k_pages must be fp8_e4m3"),
    (lambda a: a.update(v=fake([10, 16, 2, 128], ra.RL_BF16)) or a, "RL_ERR_DTYPE", "v_pages must be fp8_e4m3"),
    (lambda a: a.update(ks=None) or a, "RL_ERR_INVALID_ARG", "k_scale is NULL"),
    (lambda a: a.update(vs=fake([3], ra.RL_F32)) or a, "RL_ERR_SHAPE", "v_scale must have one entry per KV head"),
    (lambda a: a.update(ks=fake([2], ra.RL_BF16)) or a, "RL_ERR_DTYPE", "k_scale must be f32"),
    (lambda a: a.update(ks=fake([2, 1], ra.RL_F32)) or a, "RL_ERR_SHAPE", "k_scale must have 1"),
    (lambda a: a.update(vs=fake([2], ra.RL_F32, ptr=0)) or a, "RL_ERR_INVALID_ARG", "v_scale.data"),
])
def test_fp8_validation(mutate, code, needle):
    rc = call_decode_fp8(mutate(fp8_decode_args()))
    assert ra.STATUS[rc] == code, ra.last_error()
    assert needle in ra.last_error(), ra.last_error()


def test_fp8_pages_rejected_by_bf16_calls():
    a = fp8_decode_args()
    assert ra.STATUS[call_decode(a)] == "RL_ERR_DTYPE" and "k_pages must be bf16" in ra.last_error()


def test_fp8_extend_validation():
    r = ctypes.byref
    B = 3
    q = fake([10, 8, 128], ra.RL_BF16)
    k = fake([20, 16, 2, 128], ra.RL_FP8_E4M3)
    bt = fake([B, 4], ra.RL_I32)
    kv = fake([B], ra.RL_I32)
    out = fake([10, 8, 128], ra.RL_BF16)
    indptr = fake([B + 1], ra.RL_I32)
    ks = fake([2], ra.RL_F32)
    rc = ra.lib().rl_attn_extend_fp8(r(q), r(indptr), r(k), r(k), r(ks), r(fake([1], ra.RL_F32)), r(bt), r(kv),
                                     ctypes.c_float(1.0), r(out), None, None, None)
    assert ra.STATUS[rc] == "RL_ERR_SHAPE" and "v_scale" in ra.last_error()
    rc = ra.lib().rl_attn_extend_fp8(r(q), r(indptr), r(fake([20, 16, 2, 128], ra.RL_BF16)), r(k), r(ks), r(ks),
                                     r(bt), r(kv), ctypes.c_float(1.0), r(out), None, None, None)
    assert ra.STATUS[rc] == "RL_ERR_DTYPE"


def test_append_validation():
    r = ctypes.byref
    lib = ra.lib()
    B, T = 3, 10
    kn = fake([T, 2, 128], ra.RL_BF16)
    kp = fake([20, 16, 2, 128], ra.RL_BF16)
    bt = fake([B, 4], ra.RL_I32)
    kv = fake([B], ra.RL_I32)
    ind = fake([B + 1], ra.RL_I32)

    def call(k_new=kn, v_new=kn, indptr=ind, pages=kp):
        return ra.STATUS[lib.rl_attn_append_kv(r(k_new), r(v_new), r(indptr), r(bt), r(kv), r(pages), r(pages), None)]

    assert call(v_new=fake([T, 2, 64], ra.RL_BF16)) == "RL_ERR_SHAPE"
    assert call(k_new=fake([T, 2, 128], ra.RL_F32), v_new=fake([T, 2, 128], ra.RL_F32)) == "RL_ERR_DTYPE"
    assert call(k_new=fake([T, 4, 128], ra.RL_BF16), v_new=fake([T, 4, 128], ra.RL_BF16)) == "RL_ERR_SHAPE"
    assert "KV heads" in ra.last_error()
    assert call(indptr=fake([B], ra.RL_I32)) == "RL_ERR_SHAPE" and "qo_indptr" in ra.last_error()
    assert call(pages=fake([20, 16, 2, 128], ra.RL_FP8_E4M3)) == "RL_ERR_DTYPE"
    f8 = fake([20, 16, 2, 128], ra.RL_FP8_E4M3)
    sc = fake([2], ra.RL_F32)
    rc = lib.rl_attn_append_kv_fp8(r(kn), r(kn), r(ind), r(bt), r(kv), r(f8), r(f8), r(sc), r(fake([3], ra.RL_F32)), None)
    assert ra.STATUS[rc] == "RL_ERR_SHAPE" and "v_scale" in ra.last_error()
    rc = lib.rl_attn_append_kv_fp8(r(kn), r(kn), r(ind), r(bt), r(kv), r(kp), r(kp), r(sc), r(sc), None)
    assert ra.STATUS[rc] == "RL_ERR_DTYPE"
    empty = fake([0, 2, 128], ra.RL_BF16)
    assert call(k_new=empty, v_new=empty) == "RL_OK"


def test_missing_library_fails_loudly(tmp_path):
    """With no built library the binding raises instead of computing anything itself."""
    import subprocess
    import sys

    code = ("import torch\n"
            "from paper_2609_08368_amd import rl_attn as ra\n"
            "try:\n"
            "    ra.decode(torch.zeros(1, 2, 128, dtype=torch.bfloat16), torch.zeros(1, 16, 1, 128, dtype=torch.bfloat16),\n"
            "              torch.zeros(1, 16, 1, 128, dtype=torch.bfloat16), torch.zeros(1, 1, dtype=torch.int32),\n"
            "              torch.ones(1, dtype=torch.int32), 0.088)\n"
            "except RuntimeError as e:\n"
            "    print('raised:', e)\n"
            "    raise SystemExit(0)\n"
            "raise SystemExit(1)\n")
    env = dict(os.environ, RL_ATTN_LIB=str(tmp_path / "absent.so"))
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "is not built" in r.stdout, r.stdout + r.stderr
