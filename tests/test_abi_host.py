"""The C-ABI library without a GPU: it loads, exports every declared entry point,
and its host-side checks (configuration, arguments, state) return the documented
status codes before any GPU call is made."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_24204_amd import binding, configs, inputs
from tests.helpers import small_cfg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(not os.path.exists(binding.LIB_PATH),
                                reason="libwici.so not built")


def test_every_declared_symbol_is_exported():
    lib = binding.load_library()
    header = open(os.path.join(ROOT, "include", "wici.h")).read()
    declared = set(re.findall(r"\b(wici_[a-z0-9_]+)\s*\(", header))
    assert declared == set(binding.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def _cfg(**kw):
    return binding.make_config(small_cfg(d_model=256, n_heads=4, n_kv_heads=2, head_dim=64,
                                         ffn_dim=512, vocab=1000, **kw))


@pytest.mark.parametrize("name", list(configs.CONFIGS))
def test_memory_requirements_cover_the_weights(name):
    cfg = configs.CONFIGS[name]
    w, kv, s = binding.memory_requirements(binding.make_config(cfg))
    assert w >= cfg.n_params() * cfg.wbytes
    assert w < cfg.n_params() * cfg.wbytes * 1.01 + (64 << 20)
    per_pos = cfg.n_layers * 2 * cfg.kv_dim * cfg.kvbytes
    assert kv >= cfg.max_seq * per_pos
    assert all(v % 256 == 0 for v in (w, kv, s))


@pytest.mark.parametrize("field,value", [
    ("head_dim", 96), ("d_model", 100), ("ffn_dim", 96 + 1), ("n_kv_heads", 3),
    ("n_layers", 0), ("vocab", 0), ("kv_page", 48), ("prefill_chunk", 0),
    ("max_seq", 0), ("max_seq", 16385), ("rms_eps", 0.0), ("rope_base", 1.0),
    ("prefill_mode", 7),
    ("flags", 8), ("weight_dtype", 5), ("tied_embeddings", 2)])
def test_invalid_config_is_rejected(field, value):
    lib = binding.load_library()
    c = _cfg()
    setattr(c, field, value)
    h = ctypes.c_void_p()
    assert lib.wici_create(ctypes.byref(c), None, ctypes.byref(h)) == binding.WICI_E_ARG
    assert not h.value
    sz = ctypes.c_size_t()
    assert lib.wici_memory_requirements(ctypes.byref(c), ctypes.byref(sz), ctypes.byref(sz),
                                        ctypes.byref(sz)) == binding.WICI_E_ARG


@pytest.mark.parametrize("flags", [binding.WICI_FLAG_NO_GRAPH, binding.WICI_FLAG_FAULT_DRILL,
                                   binding.WICI_FLAG_NO_GRAPH | binding.WICI_FLAG_FAULT_DRILL])
def test_known_flags_are_accepted(flags):
    lib = binding.load_library()
    c = _cfg()
    c.flags = flags
    sz = ctypes.c_size_t()
    assert lib.wici_memory_requirements(ctypes.byref(c), ctypes.byref(sz), ctypes.byref(sz),
                                        ctypes.byref(sz)) == binding.WICI_OK
    assert binding.make_config(configs.TINY, fault_drill=True).flags == binding.WICI_FLAG_FAULT_DRILL


@pytest.mark.parametrize("mode,planes,ok", [
    ("bf16x3", 0x9e, True), ("bf16x3", 0xff, True), ("bf16x3", 0x55, True),
    ("bf16x3", 0x9c, False), ("bf16x3", 0x29e, True), ("bf16x3", 0x455, False),
    ("bf16x3q", 0x9e, False),
    ("bf16x2", 0x55, False)])
def test_prefill_planes_field(mode, planes, ok):
    """Two bits per product (Q/K/V, O, gate/up, down), each 1..3, two more for
    the attention's terms (0 = three), and only with the three-term mode that
    stores all of them."""
    lib = binding.load_library()
    c = _cfg(weight_dtype="bf16", kv_dtype="bf16")
    c.prefill_mode = binding.PREFILL_MODES[mode]
    c.prefill_planes = planes
    sz = ctypes.c_size_t()
    st = lib.wici_memory_requirements(ctypes.byref(c), ctypes.byref(sz), ctypes.byref(sz),
                                      ctypes.byref(sz))
    assert st == (binding.WICI_OK if ok else binding.WICI_E_ARG)


def test_make_config_packs_plane_fields():
    c = binding.make_config(configs.CONFIGS["1b"], prefill_mode="bf16x3", prefill_planes=(3, 2, 1, 2))
    assert c.prefill_planes == 3 | 2 << 2 | 1 << 4 | 2 << 6
    c = binding.make_config(configs.CONFIGS["1b"], prefill_mode="bf16x3",
                            prefill_planes=(3, 2, 2, 2, 2))
    assert c.prefill_planes == 3 | 2 << 2 | 2 << 4 | 2 << 6 | 2 << 8
    assert binding.make_config(configs.CONFIGS["1b"]).prefill_mode == binding.PREFILL_MODES["bf16x3q"]


def test_group_limit_and_fp32_weights_need_fp32_prefill():
    lib = binding.load_library()
    h = ctypes.c_void_p()
    c = _cfg(); c.n_heads, c.n_kv_heads = 18, 2
    assert lib.wici_create(ctypes.byref(c), None, ctypes.byref(h)) == binding.WICI_E_ARG
    c = _cfg(); c.weight_dtype = binding.WICI_F32; c.prefill_mode = binding.PREFILL_MODES["bf16x2"]
    assert lib.wici_create(ctypes.byref(c), None, ctypes.byref(h)) == binding.WICI_E_ARG


def test_state_machine_before_memory_is_bound():
    lib = binding.load_library()
    c = _cfg()
    h = ctypes.c_void_p()
    assert lib.wici_create(ctypes.byref(c), None, ctypes.byref(h)) == binding.WICI_OK
    try:
        pos = ctypes.c_int32(-1)
        assert lib.wici_position(h, ctypes.byref(pos)) == binding.WICI_OK and pos.value == 0
        assert lib.wici_load_weights(h, None, 0) == binding.WICI_E_STATE
        assert b"bind" in lib.wici_last_error(h)
        toks = (ctypes.c_int32 * 3)(1, 2, 3)
        out = ctypes.c_int32()
        # argument checks come first ...
        assert lib.wici_prefill(h, toks, 0, ctypes.byref(out), None) == binding.WICI_E_ARG
        bad = (ctypes.c_int32 * 2)(1, 1000)
        assert lib.wici_prefill(h, bad, 2, ctypes.byref(out), None) == binding.WICI_E_ARG
        assert lib.wici_prefill(h, toks, 3, None, None) == binding.WICI_E_ARG
        # ... then the state checks
        assert lib.wici_prefill(h, toks, 3, ctypes.byref(out), None) == binding.WICI_E_STATE
        assert lib.wici_decode_step(h, -1, ctypes.byref(out), None) == binding.WICI_E_STATE
        assert lib.wici_decode_step(h, 1000, ctypes.byref(out), None) == binding.WICI_E_ARG
        gen = (ctypes.c_int32 * 4)()
        done = ctypes.c_int32(7)
        assert lib.wici_decode_n(h, -1, 4, gen, None, None) == binding.WICI_E_ARG
        assert lib.wici_decode_n(h, -1, 0, gen, ctypes.byref(done), None) == binding.WICI_E_ARG
        assert done.value == 0
        assert lib.wici_decode_n(h, 1000, 4, gen, ctypes.byref(done), None) == binding.WICI_E_ARG
        assert lib.wici_decode_n(h, -1, 4, gen, ctypes.byref(done), None) == binding.WICI_E_STATE
        assert lib.wici_reset_kv(h) == binding.WICI_E_STATE
        buf = (ctypes.c_uint16 * 64)()
        assert lib.wici_read_kv(h, 0, 0, 1, buf, buf) == binding.WICI_E_STATE
        assert lib.wici_bind_memory(h, None, 0, None, 0, None, 0) == binding.WICI_E_ARG
        # a region that is too small is refused before anything is touched
        w, k, s = binding.memory_requirements(c)
        fake = ctypes.c_void_p(1 << 20)
        assert lib.wici_bind_memory(h, fake, w - 256, fake, k, fake, s) == binding.WICI_E_ARG
        misaligned = ctypes.c_void_p((1 << 20) + 8)
        assert lib.wici_bind_memory(h, misaligned, w, fake, k, fake, s) == binding.WICI_E_ARG
        assert lib.wici_position(h, None) == binding.WICI_E_ARG
    finally:
        lib.wici_destroy(h)
    lib.wici_destroy(None)
    assert lib.wici_create(ctypes.byref(c), None, None) == binding.WICI_E_ARG
    assert lib.wici_create(None, None, ctypes.byref(h)) == binding.WICI_E_ARG


def test_tensor_array_marshalling():
    import numpy as np
    cfg = small_cfg(d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn_dim=512, vocab=100,
                    weight_dtype="bf16", kv_dtype="bf16")
    w = {"tok_embeddings": np.zeros((100, 256), np.uint16), "norm": np.ones(256, np.float32)}
    arr, keep = binding.tensor_array(cfg, w)
    assert arr[0].name == b"tok_embeddings" and arr[0].dtype == binding.WICI_BF16
    assert arr[0].ndim == 2 and tuple(arr[0].shape) == (100, 256) and arr[0].on_device == 0
    assert arr[1].dtype == binding.WICI_F32 and arr[1].ndim == 1 and arr[1].shape[0] == 256


def test_library_quantiser_matches_oracle_bit_for_bit():
    """wici_quantize_q8 (host C++) against the oracle's float32 rule: identical codes
    and identical half-precision scale bits, on bf16 and float32 input, including
    ties, zero blocks, subnormal and rounding-boundary scales."""
    from oracle import quantize_q8 as oracle_q8
    rng = np.random.default_rng(11)
    w = (rng.standard_normal((48, 256)) * 0.02).astype(np.float32)
    w[0, :32] = 0.0
    w[1, 32:64] *= 1e-6                                   # subnormal half scales
    w[2, :32] = np.arange(32, dtype=np.float32) - 15.5     # exact half-way ratios
    w[3, :32] = (np.arange(32) % 7 - 3).astype(np.float32) * np.float32(2.0 ** -7)
    w[4, :32] = 1e-9                                      # scale rounds to zero
    w[5, 64:96] = rng.standard_normal(32).astype(np.float32) * 1000.0
    bits = np.empty(w.shape, np.uint16)
    inputs.f32_to_bf16_bits(w, bits)
    for src in (w, bits):
        ref_in = w if src.dtype == np.float32 else inputs.bf16_bits_to_f32(bits)
        q, d = oracle_q8(ref_in)
        codes, scales = binding.quantize_q8(src)
        assert np.array_equal(codes.astype(np.int16) - 128, q.astype(np.int16))
        assert np.array_equal(scales.view(np.uint16), d.view(np.uint16))
    # a random sweep over many magnitudes (scale rounding in every binade)
    w2 = (rng.standard_normal((64, 512)) * np.exp(rng.uniform(-20, 5, (64, 1)))).astype(np.float32)
    q, d = oracle_q8(w2)
    codes, scales = binding.quantize_q8(w2)
    assert np.array_equal(codes.astype(np.int16) - 128, q.astype(np.int16))
    assert np.array_equal(scales.view(np.uint16), d.view(np.uint16))


def test_library_quantiser_rejects_bad_input():
    lib = binding.load_library()
    buf = np.zeros((2, 64), np.float32)
    codes = np.empty((2, 64), np.uint8)
    scales = np.empty((2, 2), np.uint16)
    assert lib.wici_quantize_q8(buf.ctypes.data, binding.WICI_F32, 2, 48, codes.ctypes.data,
                                scales.ctypes.data) == binding.WICI_E_ARG
    assert lib.wici_quantize_q8(buf.ctypes.data, 7, 2, 64, codes.ctypes.data,
                                scales.ctypes.data) == binding.WICI_E_ARG
    buf[1, 5] = np.nan
    assert lib.wici_quantize_q8(buf.ctypes.data, binding.WICI_F32, 2, 64, codes.ctypes.data,
                                scales.ctypes.data) == binding.WICI_E_ARG


# MD5 test suite of RFC 1321 (appendix A.5)
RFC1321 = [
    (b"", "d41d8cd98f00b204e9800998ecf8427e"),
    (b"a", "0cc175b9c0f1b6a831c399e269772661"),
    (b"abc", "900150983cd24fb0d6963f7d28e17f72"),
    (b"message digest", "f96b697d7cb7938d525a2f31aaf161d0"),
    (b"abcdefghijklmnopqrstuvwxyz", "c3fcd3d76192e4007dfb496cca67e13b"),
    (b"ABCDEFGHIJKLMNOPQRSTUVWXYZabcdefghijklmnopqrstuvwxyz0123456789",
     "d174ab98d277d9f5a5611c2c9f419d9f"),
    (b"1234567890" * 8, "57edf4a22be3c955ac49da2e2107b67a"),
]


@pytest.mark.parametrize("msg,digest", RFC1321)
def test_md5_rfc1321_suite(msg, digest):
    assert binding.md5(np.frombuffer(msg, np.uint8)).hex() == digest


def test_md5_lengths_around_block_boundaries():
    import hashlib
    rng = np.random.default_rng(3)
    for n in [1, 55, 56, 57, 63, 64, 65, 119, 120, 127, 128, 129, 1000, 4096, 100003]:
        a = rng.integers(0, 256, n, dtype=np.uint8)
        assert binding.md5(a) == hashlib.md5(a.tobytes()).digest(), n


def test_cached_load_checks_arguments():
    lib = binding.load_library()
    out = (ctypes.c_int32 * 1)()
    assert lib.wici_load_weights_cached(None, None, None, 0, b"/tmp", 0, out) == binding.WICI_E_ARG
    c = _cfg()
    h = ctypes.c_void_p()
    assert lib.wici_create(ctypes.byref(c), None, ctypes.byref(h)) == binding.WICI_OK
    try:
        t = (binding.WiciTensor * 1)()
        t[0].name = b"norm"
        t[0].dtype = binding.WICI_F32
        t[0].ndim = 1
        t[0].shape[0] = c.d_model
        t[0].data = None
        # below the threshold a tensor must carry data
        assert lib.wici_load_weights_cached(h, t, None, 1, b"/tmp", 1 << 30, out) == binding.WICI_E_ARG
        assert lib.wici_load_weights_cached(h, t, None, 1, None, 0, out) == binding.WICI_E_ARG
        assert lib.wici_load_weights_cached(h, t, None, 1, b"/tmp", -1, out) == binding.WICI_E_ARG
    finally:
        lib.wici_destroy(h)


def test_cached_load_rejects_data_that_does_not_match_its_hash(tmp_path):
    """A store miss with both a hash and data saves the data under that hash,
    so the library hashes the data first: a wrong hash is an argument error
    (before anything is uploaded), the right one passes that check."""
    lib = binding.load_library()
    c = _cfg()
    h = ctypes.c_void_p()
    assert lib.wici_create(ctypes.byref(c), None, ctypes.byref(h)) == binding.WICI_OK
    try:
        data = np.arange(c.d_model, dtype=np.float32)
        t = (binding.WiciTensor * 1)()
        t[0].name = b"norm"
        t[0].dtype = binding.WICI_F32
        t[0].ndim = 1
        t[0].shape[0] = c.d_model
        t[0].data = data.ctypes.data
        out = (ctypes.c_int32 * 1)()
        good = binding.md5(data)
        bad = bytes([good[0] ^ 1]) + good[1:]
        store = str(tmp_path).encode()
        for digest, want in ((bad, binding.WICI_E_ARG), (good, binding.WICI_E_STATE)):
            hb = (ctypes.c_uint8 * 16).from_buffer_copy(digest)
            # threshold 0: the tensor goes through the store; the model has no
            # memory bound yet, so a hash that passes stops at the upload
            assert lib.wici_load_weights_cached(h, t, hb, 1, store, 0, out) == want
        assert not os.listdir(tmp_path)
    finally:
        lib.wici_destroy(h)

