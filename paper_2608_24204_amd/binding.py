"""ctypes binding of libwici.so (declared in include/wici.h).

Argument marshalling only: every step of the forward runs in the library's HIP
kernels.  torch is used to allocate the device regions the library binds and to
provide the HIP stream it launches on.  If the library is missing this module
raises; there is no other code path.
"""

from __future__ import annotations

import ctypes
import os
from typing import Mapping

import numpy as np

from .configs import ModelConfig

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwici.so")

WICI_OK, WICI_E_ARG, WICI_E_STATE, WICI_E_CAPACITY, WICI_E_HIP, WICI_E_NUMERIC = 0, -1, -2, -3, -4, -5
STATUS_NAMES = {0: "WICI_OK", -1: "WICI_E_ARG", -2: "WICI_E_STATE", -3: "WICI_E_CAPACITY",
                -4: "WICI_E_HIP", -5: "WICI_E_NUMERIC"}
WICI_F32, WICI_BF16, WICI_Q8 = 0, 1, 2
PREFILL_MODES = {"bf16x2": 0, "bf16": 1, "f32": 2, "bf16x3": 3, "bf16x3q": 4}
WICI_FLAG_NO_GRAPH = 1
WICI_FLAG_FAULT_DRILL = 2

# every entry point include/wici.h declares
EXPORTED = ["wici_create", "wici_memory_requirements", "wici_bind_memory", "wici_load_weights",
            "wici_prefill", "wici_decode_step", "wici_decode_n", "wici_reset_kv", "wici_position",
            "wici_read_kv", "wici_profile_decode_step", "wici_quantize_q8", "wici_md5",
            "wici_load_weights_cached", "wici_bind_memory_shared", "wici_decode_batch",
            "wici_stream_read", "wici_stream_read_noalloc", "wici_last_error", "wici_destroy"]


class WiciConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_double),
        ("tied_embeddings", ctypes.c_int32), ("weight_dtype", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32), ("max_seq", ctypes.c_int32),
        ("prefill_chunk", ctypes.c_int32), ("kv_page", ctypes.c_int32),
        ("prefill_mode", ctypes.c_int32), ("flags", ctypes.c_int32),
        ("prefill_planes", ctypes.c_int32),
    ]


class WiciTensor(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 2), ("data", ctypes.c_void_p),
                ("on_device", ctypes.c_int32)]


class WiciError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_lib = None


def load_library(path: str | None = None) -> ctypes.CDLL:
    """Load libwici.so and declare its signatures (raises if it was not built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise FileNotFoundError(f"{p} not found: build it with `python -m paper_2608_24204_amd.build`")
    lib = ctypes.CDLL(p)
    P = ctypes.c_void_p
    i32, sz = ctypes.c_int32, ctypes.c_size_t
    sig = {
        "wici_create": ([ctypes.POINTER(WiciConfig), P, ctypes.POINTER(P)], ctypes.c_int),
        "wici_memory_requirements": ([ctypes.POINTER(WiciConfig), ctypes.POINTER(sz),
                                      ctypes.POINTER(sz), ctypes.POINTER(sz)], ctypes.c_int),
        "wici_bind_memory": ([P, P, sz, P, sz, P, sz], ctypes.c_int),
        "wici_load_weights": ([P, ctypes.POINTER(WiciTensor), i32], ctypes.c_int),
        "wici_prefill": ([P, P, i32, ctypes.POINTER(i32), P], ctypes.c_int),
        "wici_decode_step": ([P, i32, ctypes.POINTER(i32), P], ctypes.c_int),
        "wici_decode_n": ([P, i32, i32, P, ctypes.POINTER(i32), P], ctypes.c_int),
        "wici_reset_kv": ([P], ctypes.c_int),
        "wici_position": ([P, ctypes.POINTER(i32)], ctypes.c_int),
        "wici_read_kv": ([P, i32, i32, i32, P, P], ctypes.c_int),
        "wici_profile_decode_step": ([P, i32, ctypes.POINTER(i32), P, i32, ctypes.POINTER(i32)],
                                     ctypes.c_int),
        "wici_quantize_q8": ([P, i32, ctypes.c_int64, ctypes.c_int64, P, P], ctypes.c_int),
        "wici_md5": ([P, sz, P], ctypes.c_int),
        "wici_load_weights_cached": ([P, ctypes.POINTER(WiciTensor), P, i32, ctypes.c_char_p,
                                      ctypes.c_int64, P], ctypes.c_int),
        "wici_bind_memory_shared": ([P, P, P, sz, P, sz], ctypes.c_int),
        "wici_decode_batch": ([P, i32, P, P, P], ctypes.c_int),
        "wici_stream_read": ([P, sz, i32, i32, P, P, ctypes.POINTER(ctypes.c_float), P],
                             ctypes.c_int),
        "wici_stream_read_noalloc": ([P, sz, i32, P, ctypes.POINTER(ctypes.c_uint32)],
                                     ctypes.c_int),
        "wici_last_error": ([P], ctypes.c_char_p),
        "wici_destroy": ([P], None),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    if path is None:
        _lib = lib
    return lib


def make_config(cfg: ModelConfig, prefill_mode: str | None = None, graph: bool = True,
                max_seq: int | None = None, prefill_chunk: int | None = None,
                kv_page: int | None = None, prefill_planes=None,
                fault_drill: bool = False) -> WiciConfig:
    """prefill_planes: None/0 for prefill_mode's own term count, or a tuple
    (qkv, o, gate_up, down[, attention]) of bf16 terms each projection reads and
    the prefill attention carries (bf16x3 only; attention defaults to three)."""
    if prefill_mode is None:
        prefill_mode = "f32" if cfg.weight_dtype == "f32" else "bf16x3q"
    c = WiciConfig()
    c.n_layers, c.d_model, c.n_heads = cfg.n_layers, cfg.d_model, cfg.n_heads
    c.n_kv_heads, c.head_dim, c.ffn_dim, c.vocab = cfg.n_kv_heads, cfg.head_dim, cfg.ffn_dim, cfg.vocab
    c.rms_eps, c.rope_base = cfg.rms_eps, cfg.rope_base
    c.tied_embeddings = int(cfg.tied_embeddings)
    c.weight_dtype = {"bf16": WICI_BF16, "f32": WICI_F32, "q8": WICI_Q8}[cfg.weight_dtype]
    c.kv_dtype = WICI_BF16 if cfg.kv_dtype == "bf16" else WICI_F32
    c.max_seq = cfg.max_seq if max_seq is None else max_seq
    c.prefill_chunk = cfg.prefill_chunk if prefill_chunk is None else prefill_chunk
    c.kv_page = cfg.kv_page if kv_page is None else kv_page
    c.prefill_mode = PREFILL_MODES[prefill_mode]
    c.flags = (0 if graph else WICI_FLAG_NO_GRAPH) | (WICI_FLAG_FAULT_DRILL if fault_drill else 0)
    if prefill_planes:
        q, o, gu, dn, *at = prefill_planes
        c.prefill_planes = q | (o << 2) | (gu << 4) | (dn << 6) | ((at[0] if at else 0) << 8)
    return c


def quantize_q8(w: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """The library's host quantiser (wici_quantize_q8) on a float32 or bf16-bits
    (uint16) matrix [rows, cols]: returns (codes uint8 = q + 128, scales as float16)."""
    lib = load_library()
    w = np.ascontiguousarray(w)
    dt = WICI_BF16 if w.dtype == np.uint16 else WICI_F32
    if dt == WICI_F32:
        w = np.ascontiguousarray(w, dtype=np.float32)
    rows, cols = w.shape
    codes = np.empty((rows, cols), np.uint8)
    scales = np.empty((rows, cols // 32), np.uint16)
    st = lib.wici_quantize_q8(w.ctypes.data, dt, rows, cols, codes.ctypes.data, scales.ctypes.data)
    if st != WICI_OK:
        raise WiciError(st, "wici_quantize_q8")
    return codes, scales.view(np.float16)


WICI_CACHE_SENT, WICI_CACHE_HIT, WICI_CACHE_SAVED, WICI_CACHE_NEEDED = 0, 1, 2, 3


def md5(data) -> bytes:
    """The library's MD5 (wici_md5) of a numpy array's bytes."""
    lib = load_library()
    a = np.ascontiguousarray(data)
    out = (ctypes.c_uint8 * 16)()
    st = lib.wici_md5(a.ctypes.data if a.nbytes else None, a.nbytes, out)
    if st != WICI_OK:
        raise WiciError(st, "wici_md5")
    return bytes(out)


def stream_read(buf, grid: int, reps: int, sink, stream=None, checksum: bool = False):
    """One plain streaming read of the device tensor ``buf`` by ``grid`` workgroups,
    ``reps`` times (wici_stream_read): returns the average ms per read, and with
    ``checksum`` also the XOR of the buffer's 32-bit words.  ``sink`` is a device
    tensor of at least 4 * (256 * grid + 1) bytes; ``stream`` a torch stream
    (default: the current one)."""
    import torch
    lib = load_library()
    st = (stream or torch.cuda.current_stream()).cuda_stream
    if sink.numel() * sink.element_size() < 4 * (256 * grid + 1):
        raise ValueError("sink too small")
    ms = ctypes.c_float()
    ck = ctypes.c_uint32()
    r = lib.wici_stream_read(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
                             grid, reps, ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(st),
                             ctypes.byref(ms), ctypes.byref(ck) if checksum else None)
    if r != WICI_OK:
        raise WiciError(r, "wici_stream_read failed")
    return (float(ms.value), int(ck.value)) if checksum else float(ms.value)


def memory_requirements(c: WiciConfig) -> tuple[int, int, int]:
    lib = load_library()
    w, k, s = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    st = lib.wici_memory_requirements(ctypes.byref(c), ctypes.byref(w), ctypes.byref(k), ctypes.byref(s))
    if st != WICI_OK:
        raise WiciError(st, "invalid configuration")
    return w.value, k.value, s.value


def tensor_array(cfg: ModelConfig, weights: Mapping[str, object]):
    """Build the wici_tensor array for numpy (host) or torch (device) arrays.
    Returns (array, keepalive list)."""
    arr = (WiciTensor * len(weights))()
    keep = []
    for i, (name, a) in enumerate(weights.items()):
        t = arr[i]
        nb = name.encode()
        keep.append(nb)
        t.name = nb
        if isinstance(a, np.ndarray):
            a = np.ascontiguousarray(a)
            keep.append(a)
            t.data = a.ctypes.data
            t.on_device = 0
            dt = a.dtype
            shape = a.shape
            t.dtype = WICI_BF16 if dt == np.uint16 else WICI_F32
            if dt not in (np.uint16, np.float32):
                raise TypeError(f"{name}: dtype {dt} (bf16 bits as uint16 or float32)")
        else:  # a torch tensor on the model's device
            import torch
            a = a.contiguous()
            keep.append(a)
            t.data = a.data_ptr()
            t.on_device = 1 if a.is_cuda else 0
            shape = tuple(a.shape)
            if a.dtype in (torch.bfloat16, torch.uint16, torch.int16):
                t.dtype = WICI_BF16
            elif a.dtype == torch.float32:
                t.dtype = WICI_F32
            else:
                raise TypeError(f"{name}: dtype {a.dtype}")
        t.ndim = len(shape)
        t.shape[0] = shape[0]
        t.shape[1] = shape[1] if len(shape) > 1 else 0
    return arr, keep


class WiciModel:
    """One model on one GPU: owns the device regions (torch allocations) and the
    library handle."""

    def __init__(self, cfg: ModelConfig, *, prefill_mode: str | None = None, graph: bool = True,
                 max_seq: int | None = None, prefill_chunk: int | None = None,
                 kv_page: int | None = None, device: int = 0,
                 share_weights_of: "WiciModel | None" = None, prefill_planes=None,
                 fault_drill: bool = False):
        """share_weights_of: another (loaded) model whose weights this one uses
        (wici_bind_memory_shared); only the KV cache and scratch are allocated.
        prefill_planes: see make_config.  fault_drill: WICI_FLAG_FAULT_DRILL
        (tests of the misplaced-split error path)."""
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("WiciModel needs a HIP GPU")
        self.cfg = cfg
        self.lib = load_library()
        self.device = torch.device("cuda", device)
        self.c = make_config(cfg, prefill_mode, graph, max_seq, prefill_chunk, kv_page,
                             prefill_planes, fault_drill)
        wb, kb, sb = memory_requirements(self.c)
        self.mem_bytes = (wb, kb, sb)
        self.stream = torch.cuda.Stream(self.device)
        self._src = share_weights_of
        self._w = None if share_weights_of is not None else \
            torch.empty(wb, dtype=torch.uint8, device=self.device)
        self._kv = torch.empty(kb, dtype=torch.uint8, device=self.device)
        self._s = torch.empty(sb, dtype=torch.uint8, device=self.device)
        torch.cuda.synchronize(self.device)
        h = ctypes.c_void_p()
        self._check(self.lib.wici_create(ctypes.byref(self.c), ctypes.c_void_p(self.stream.cuda_stream),
                                         ctypes.byref(h)), "wici_create", handle=None)
        self.h = h
        if share_weights_of is not None:
            self._check(self.lib.wici_bind_memory_shared(self.h, share_weights_of.h,
                                                         self._kv.data_ptr(), kb,
                                                         self._s.data_ptr(), sb),
                        "wici_bind_memory_shared")
        else:
            self._check(self.lib.wici_bind_memory(self.h, self._w.data_ptr(), wb, self._kv.data_ptr(),
                                                  kb, self._s.data_ptr(), sb), "wici_bind_memory")
        self._logits = np.empty(cfg.vocab, np.float32)
        # per-step call state, built once (the greedy loop calls decode_step per token)
        self._tok = ctypes.c_int32()
        self._tok_ref = ctypes.byref(self._tok)
        self._decode_step_fn = self.lib.wici_decode_step

    def _check(self, st: int, what: str, handle="self"):
        if st != WICI_OK:
            msg = what
            if handle == "self" and getattr(self, "h", None):
                msg = f"{what}: {self.lib.wici_last_error(self.h).decode()}"
            raise WiciError(st, msg)

    def load_weights(self, weights: Mapping[str, object]) -> None:
        arr, keep = tensor_array(self.cfg, weights)
        self._check(self.lib.wici_load_weights(self.h, arr, len(weights)), "wici_load_weights")
        del keep

    def load_weights_cached(self, weights: Mapping[str, object], store_dir: str,
                            threshold_bytes: int = 0, hashes: Mapping[str, bytes] | None = None):
        """Upload through the content store (wici_load_weights_cached).  With `hashes`
        (name -> 16-byte MD5), tensors named there are sent as hashes only (no data);
        returns {name: WICI_CACHE_* outcome}."""
        names = list(weights)
        if hashes is not None:
            send = {n: (None if n in hashes else weights[n]) for n in names}
        else:
            send = weights
        arr, keep = tensor_array(self.cfg, {n: (weights[n] if send[n] is None else send[n])
                                            for n in names})
        if hashes is not None:
            for i, n in enumerate(names):
                if n in hashes:
                    arr[i].data = None
        hb = None
        if hashes is not None:
            # the library reads the hash of every tensor at or above the threshold:
            # those not given are hashed here from their data (the caller's side of
            # the exchange); smaller tensors are always sent and need none
            hb = np.zeros((len(names), 16), np.uint8)
            for i, n in enumerate(names):
                h = hashes.get(n)
                if h is None and np.asarray(weights[n]).nbytes >= threshold_bytes:
                    h = md5(weights[n])
                if h is not None:
                    hb[i] = np.frombuffer(h, np.uint8)
        out = np.zeros(len(names), np.int32)
        self._check(self.lib.wici_load_weights_cached(
            self.h, arr, hb.ctypes.data if hb is not None else None, len(names),
            store_dir.encode(), int(threshold_bytes), out.ctypes.data), "wici_load_weights_cached")
        del keep
        return {n: int(o) for n, o in zip(names, out)}

    def prefill(self, tokens, want_logits: bool = False):
        toks = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32).reshape(-1))
        out = ctypes.c_int32()
        lg = self._logits.ctypes.data if want_logits else None
        self._check(self.lib.wici_prefill(self.h, toks.ctypes.data, toks.size, ctypes.byref(out), lg),
                    "wici_prefill")
        return out.value, (self._logits.copy() if want_logits else None)

    def decode_step(self, token_in: int = -1, want_logits: bool = False):
        lg = self._logits.ctypes.data if want_logits else None
        st = self._decode_step_fn(self.h, int(token_in), self._tok_ref, lg)
        if st != WICI_OK:
            self._check(st, "wici_decode_step")
        return self._tok.value, (self._logits.copy() if want_logits else None)

    def decode_n(self, n: int, token_in: int = -1, want_logits: bool = False):
        """n greedy decode steps in one call (argmax fed back on the device).
        Returns (int32 array of n tokens, last step's logits or None).  On non-finite
        logits raises WiciError carrying `.tokens`, the steps that completed."""
        toks = np.full(max(int(n), 1), -1, np.int32)
        done = ctypes.c_int32()
        lg = self._logits.ctypes.data if want_logits else None
        st = self.lib.wici_decode_n(self.h, int(token_in), int(n), toks.ctypes.data,
                                    ctypes.byref(done), lg)
        if st == WICI_E_NUMERIC:
            err = WiciError(st, f"wici_decode_n: {self.lib.wici_last_error(self.h).decode()}")
            err.tokens = toks[:done.value].copy()
            raise err
        self._check(st, "wici_decode_n")
        return toks[:n], (self._logits.copy() if want_logits else None)

    def reset_kv(self) -> None:
        self._check(self.lib.wici_reset_kv(self.h), "wici_reset_kv")

    @property
    def position(self) -> int:
        p = ctypes.c_int32()
        self._check(self.lib.wici_position(self.h, ctypes.byref(p)), "wici_position")
        return p.value

    def read_kv(self, layer: int, begin: int, end: int):
        c = self.cfg
        dt = np.uint16 if c.kv_dtype == "bf16" else np.float32
        K = np.empty((end - begin, c.n_kv_heads, c.head_dim), dt)
        V = np.empty_like(K)
        self._check(self.lib.wici_read_kv(self.h, layer, begin, end, K.ctypes.data, V.ctypes.data),
                    "wici_read_kv")
        return K, V

    def profile_decode_step(self, token_in: int = -1):
        """One eager decode step with per-launch HIP-event durations (ms), in the
        order embed, per layer (qkv, attention, o, gate/up, down), lm_head, argmax."""
        n = 3 + 5 * self.cfg.n_layers
        dur = np.zeros(n, np.float32)
        out, nw = ctypes.c_int32(), ctypes.c_int32()
        self._check(self.lib.wici_profile_decode_step(self.h, int(token_in), ctypes.byref(out),
                                                      dur.ctypes.data, n, ctypes.byref(nw)),
                    "wici_profile_decode_step")
        return out.value, dur[:nw.value]

    def generate(self, prompt, n_steps: int, want_logits: bool = False):
        """Greedy run: prefill then n_steps decode steps feeding back each token."""
        tok, lg = self.prefill(prompt, want_logits)
        ids, logs = [tok], [lg]
        for _ in range(n_steps):
            tok, lg = self.decode_step(-1, want_logits)
            ids.append(tok)
            logs.append(lg)
        return ids, logs

    @staticmethod
    def decode_batch(models, tokens_in=None, want_logits: bool = False):
        """One greedy step for several models sharing weights (wici_decode_batch);
        returns the next token of each (and their logits [n, vocab] if asked)."""
        n = len(models)
        arr = (ctypes.c_void_p * n)(*[m.h.value if isinstance(m.h, ctypes.c_void_p) else m.h
                                      for m in models])
        toks = None
        if tokens_in is not None:
            toks = np.ascontiguousarray(np.asarray(tokens_in, np.int32))
        out = np.zeros(n, np.int32)
        lg = np.empty((n, models[0].cfg.vocab), np.float32) if want_logits else None
        lead = models[0]
        lead._check(lead.lib.wici_decode_batch(arr, n, toks.ctypes.data if toks is not None else None,
                                               out.ctypes.data,
                                               lg.ctypes.data if lg is not None else None),
                    "wici_decode_batch")
        return (out, lg) if want_logits else out

    def close(self) -> None:
        if getattr(self, "h", None):
            self.lib.wici_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
