"""CPU-only checks of the C ABI: the library loads, exports what sbd.h declares, and rejects
bad arguments on the host before touching a GPU."""
import ctypes
import math
import os
import re

import pytest

import synth
import paper_2509_04185_amd as P
from paper_2509_04185_amd import binding as Bd

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "sbd.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sbd_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    return P.load_library()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(Bd.SIGNATURES) == names


def test_status_strings(lib):
    for s in range(7):
        assert lib.sbd_status_string(s)
    assert P.status_string(3) == "capacity exceeded"


def test_config_struct_matches_header():
    src = open(HEADER).read()
    m = re.search(r"typedef struct \{(.*?)\} sbd_model_config;", src, re.S)
    fields = re.findall(r"\b([a-z_]+)\s*[,;]", re.sub(r"(int32_t|float)", "", m.group(1)))
    assert [f for f, _ in Bd.ModelConfig._fields_] == fields


@pytest.mark.parametrize("name", sorted(synth.WORKLOADS))
def test_workspace_bytes_for_every_workload(name):
    w = synth.WORKLOADS[name]
    cfg = P.make_config(w.shape, w.batch, max(w.cache_lens()) + 64, w.k)
    n = P.workspace_bytes(cfg)
    s = w.shape
    cap = (max(w.cache_lens()) + 64 + 63) // 64 * 64
    kv = 2 * s.n_layers * w.batch * s.n_kv_heads * cap * s.head_dim * 2
    qd, kvd, d, F = s.n_q_heads * s.head_dim, s.n_kv_heads * s.head_dim, s.d_model, s.ffn_dim
    weights = 2 * (s.n_layers * ((qd + 2 * kvd) * d + d * qd + 3 * F * d) + s.vocab * d)
    assert kv + weights < n < kv + weights + 2 * 2**30


@pytest.mark.parametrize("field,value", [("head_dim", 96), ("d_model", 200), ("vocab", 1000),
                                         ("n_kv_heads", 3), ("max_block", 65), ("mask_id", 1024),
                                         ("max_batch", 0), ("ffn_dim", 100), ("qk_norm", 2)])
def test_unsupported_configs_are_rejected(field, value):
    cfg = P.make_config(synth.TINY, 1, 128, 4)
    setattr(cfg, field, value)
    with pytest.raises(P.SbdError) as e:
        P.workspace_bytes(cfg)
    assert e.value.name == "SBD_ERR_UNSUPPORTED"


def test_unknown_weight_format_rejected():
    cfg = P.make_config(synth.TINY, 1, 64, 4)
    cfg.weight_format = 2
    with pytest.raises(P.SbdError, match="weight_format"):
        P.workspace_bytes(cfg)


def test_kv_format_checks_and_workspace():
    """An e4m3 KV cache takes one byte per element; unknown formats and out-of-range scale
    exponents are rejected (the exponent is ignored with a bf16 cache)."""
    s = synth.LLAMA8B
    b16 = P.workspace_bytes(P.make_config(s, 2, 4096, 16))
    b8 = P.workspace_bytes(P.make_config(s, 2, 4096, 16, kv_format="fp8_e4m3", kv_scale_exp=-4))
    kv_elems = 2 * s.n_layers * 2 * s.n_kv_heads * 4096 * s.head_dim   # K and V
    assert b16 - b8 == pytest.approx(kv_elems, abs=1024)
    for fmt, exp in ((2, 0), (1, 101), (1, -101)):
        cfg = P.make_config(synth.TINY, 1, 64, 4)
        cfg.kv_format, cfg.kv_scale_exp = fmt, exp
        with pytest.raises(P.SbdError, match="kv_"):
            P.workspace_bytes(cfg)
    cfg = P.make_config(synth.TINY, 1, 64, 4)
    cfg.kv_scale_exp = 500
    assert P.workspace_bytes(cfg) > 0


def test_fp8_workspace_holds_both_packings():
    """FP8 weights: the e4m3 packing (1 byte per element) and the widened bf16 copy."""
    s = synth.LLAMA8B
    b16 = P.workspace_bytes(P.make_config(s, 1, 2112, 16))
    f8 = P.workspace_bytes(P.make_config(s, 1, 2112, 16, weight_format="fp8_e4m3"))
    qd, kvd, d, F = s.n_q_heads * s.head_dim, s.n_kv_heads * s.head_dim, s.d_model, s.ffn_dim
    elems = s.n_layers * ((qd + 2 * kvd) * d + d * qd + 3 * F * d) + s.vocab * d
    assert elems <= f8 - b16 <= elems + 64 * 2**20


def test_bad_eps_and_theta_rejected():
    for field, value in (("rms_eps", 0.0), ("rms_eps", math.nan), ("rope_theta", -1.0)):
        cfg = P.make_config(synth.TINY, 1, 128, 4)
        setattr(cfg, field, value)
        with pytest.raises(P.SbdError):
            P.workspace_bytes(cfg)


def test_create_argument_errors(lib):
    cfg = P.make_config(synth.TINY, 1, 128, 4)
    out = ctypes.c_void_p()
    w = Bd.Weights()
    st = lib.sbd_create(ctypes.byref(cfg), ctypes.byref(w), None, 0, None, ctypes.byref(out))
    assert st == 1 and out.value is None
    assert b"workspace" in lib.sbd_last_error(None)
    # misaligned workspace
    st = lib.sbd_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.c_void_p(0x1001), 1 << 40, None,
                        ctypes.byref(out))
    assert st == 1 and b"aligned" in lib.sbd_last_error(None)
    # too small
    st = lib.sbd_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.c_void_p(0x100000), 16, None,
                        ctypes.byref(out))
    assert st == 4
    # null weights
    st = lib.sbd_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.c_void_p(0x100000), 1 << 40, None,
                        ctypes.byref(out))
    assert st == 1 and b"weight" in lib.sbd_last_error(None)


def test_null_context_is_rejected(lib):
    assert lib.sbd_eb_select(None, 1, 4, 32, None, None, 0.5, -1, None, None, None, None) == 1
    assert lib.sbd_select(None, 1, 1, 4, 32, None, None, 0.5, -1, None, None, None, None, None) == 1
    assert lib.sbd_block_forward(None, 1, None, 4, None, None, None, None, None) == 1
    assert lib.sbd_commit(None, 1, None, None) == 1
    assert lib.sbd_block_step(None, 0, 1, None, 4, None, None, None, None, 1.0, None, None, None, None, None,
                              None) == 1
    assert lib.sbd_prefill(None, 0, None, 1, None) == 1
    assert lib.sbd_destroy(None) == 1
    assert lib.sbd_set_decode_path(None, 0) == 1
    assert lib.sbd_kv_import(None, 0, 0, 1, None, None) == 1
    n = ctypes.c_int32()
    assert lib.sbd_cache_len(None, 0, ctypes.byref(n)) == 1


def test_noalloc_eb_select_validates_before_any_device_call(lib):
    """Sizes beyond the static scratch and bad arguments are refused on the host (no GPU here)."""
    d = ctypes.c_void_p(16)   # never dereferenced: every case fails validation first
    m = (ctypes.c_uint8 * 2048)()
    f = lib.sbd_eb_select_noalloc
    assert f(None, 17, 64, 128, d, m, 1.0, -1, d, d, d, None) == 1          # 1088 rows
    assert f(None, 1, 65, 128, d, m, 1.0, -1, d, d, d, None) == 1           # k > 64
    assert f(None, 1, 4, 262145, d, m, 1.0, -1, d, d, d, None) == 1         # vocab > 64 chunks
    assert f(None, 1, 4, 128, None, m, 1.0, -1, d, d, d, None) == 1         # null logits
    assert f(None, 1, 4, 128, d, m, float("nan"), -1, d, d, d, None) == 1   # NaN gamma
    assert f(None, 1, 4, 128, d, m, 1.0, 128, d, d, d, None) == 1           # mask id out of range
    assert b"static scratch" in lib.sbd_last_error(None) or b"mask_id" in lib.sbd_last_error(None)


def test_xcd_map_decision():
    """The check behind the per-XCD kernels' placement assumption: workgroup i on XCD i % n."""
    f = P.load_library().sbd_xcd_map_check
    ok = ctypes.c_int32(-1)

    def check(ids, n_xcd=8):
        arr = (ctypes.c_int32 * len(ids))(*ids)
        assert f(arr, len(ids), n_xcd, ctypes.byref(ok)) == 0
        return ok.value

    assert check([i % 8 for i in range(2048)]) == 1
    assert check([(i + 1) % 8 for i in range(256)]) == 0           # shifted by one XCD
    assert check([(i // 32) for i in range(256)]) == 0             # blocks of 32 per XCD
    ids = [i % 8 for i in range(1000)]
    ids[999] = 0
    assert check(ids) == 0                                          # one misplaced workgroup
    assert check([0] * 64, n_xcd=1) == 1
    assert f(None, 4, 8, ctypes.byref(ok)) == 1


def test_workspace_regions():
    cfg = P.make_config(synth.TINY, 1, 128, 4)
    total = P.workspace_bytes(cfg)
    lib = P.load_library()
    for name in Bd.Sbd.REGION_DTYPES:
        off, nb = ctypes.c_size_t(), ctypes.c_size_t()
        assert lib.sbd_workspace_region(ctypes.byref(cfg), name.encode(), ctypes.byref(off),
                                        ctypes.byref(nb)) == 0
        assert off.value % 256 == 0 and off.value + nb.value <= total
    off, nb = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.sbd_workspace_region(ctypes.byref(cfg), b"nope", ctypes.byref(off), ctypes.byref(nb)) == 1
