"""Thin Python binding of the Kraken C ABI (include/kraken.h).

Argument marshalling only: every step of the prefill runs in the HIP kernels of
``libkraken.so``.  torch provides device memory and the current stream.  If the
library has not been built this module raises instead of falling back to
anything else.
"""

from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Iterable, List, Mapping, Optional, Sequence, Tuple

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkraken.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_OOM, ERR_STATE, ERR_HIP, ERR_OVERFLOW = range(7)
DTYPE_F32, DTYPE_BF16, DTYPE_F16 = 0, 1, 2
COMPUTE_CODES = {"storage": 0, "f32": 1, "bf16": 2, "f16": 3}
MAX_SEQS = 256
# floats of the static scratch of kraken_op_decode_attention_noalloc (kraken.h)
NOALLOC_SCRATCH_FLOATS = 8 * 1024 * 1024

ARCH_CODES = {"kraken": 0, "gpt": 1, "parallel": 2}

# kernel classes of the per-kernel timer (kraken.h)
K_LN1, K_GEMM_QK, K_GEMM_VT, K_ATTN, K_GEMM_O, K_COMBINE, K_GEMM_UP, K_GEMM_DOWN, K_CONCAT, \
    K_OTHER, K_KV, K_UNEMBED = range(12)
K_COUNT = 12
KERNEL_CLASS_NAMES = ["ln1", "gemm_qk", "gemm_vt", "attention", "gemm_o", "combine_ln2",
                      "gemm_up", "gemm_down", "w_concat", "other", "kv_cache", "unembed"]

EPI_BIAS_N, EPI_BIAS_N_GELU, EPI_BIAS_N_RES, EPI_BIAS_M = range(4)

# Order of one sub-layer's tensors in the weight blob (kraken_load_weights); the parallel
# attention + FFN layer has no ln2_g / ln2_b.  Embeddings follow the layers (and W_concat).
BLOB_ORDER = ("ln1_g", "ln1_b", "Wqkv", "bqkv", "Wo", "bo",
              "ln2_g", "ln2_b", "W1", "b1", "W2", "b2")
EMB_ORDER = ("tok_emb", "pos_emb", "lnf_g", "lnf_b")


class KrakenError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"kraken status {status}: {msg}")
        self.status = status


class _Config(ctypes.Structure):
    _fields_ = [("n_sub", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("d_ff", ctypes.c_int32), ("max_tokens", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("compute", ctypes.c_int32),
                ("ln_eps", ctypes.c_float), ("n_kv_heads", ctypes.c_int32),
                ("arch", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("max_positions", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """Loads libkraken.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2408_07802_amd.build` (or __graft_entry__.build())")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    fp = ctypes.c_float
    P = ctypes.POINTER
    sigs = {
        "kraken_create": ([P(_Config), P(vp)], i32),
        "kraken_weight_blob_elems": ([P(_Config)], sz),
        "kraken_load_weights": ([vp, vp, sz, ctypes.c_int, vp], i32),
        "kraken_prefill": ([vp, vp, P(i32), i32, vp, vp, vp], i32),
        "kraken_forward_tokens": ([vp, P(i32), P(i32), i32, vp, vp, vp], i32),
        "kraken_kv_cache_bytes": ([P(_Config), i32, i32], sz),
        "kraken_prefill_kv": ([vp, vp, P(i32), i32, vp, vp, vp, i32, i32, vp], i32),
        "kraken_decode": ([vp, vp, P(i32), i32, vp, vp, vp, i32, i32, vp], i32),
        "kraken_destroy": ([vp], i32),
        "kraken_sync": ([vp, vp], i32),
        "kraken_debug_poison_workspace": ([vp, vp], i32),
        "kraken_status_string": ([i32], ctypes.c_char_p),
        "kraken_last_error": ([], ctypes.c_char_p),
        "kraken_profile_enable": ([vp, ctypes.c_int], i32),
        "kraken_profile_read": ([vp, ctypes.c_int, P(ctypes.c_double), P(i64)], i32),
        "kraken_profile_reset": ([vp], i32),
        "kraken_class_flops": ([P(_Config), ctypes.c_int, P(i32), i32], ctypes.c_double),
        "kraken_op_layernorm": ([i32, vp, i64, vp, vp, vp, i32, i32, i32, fp, vp], i32),
        "kraken_op_combine_ln2": ([i32, vp, vp, vp, vp, vp, vp, i32, i32, i32, fp, vp], i32),
        "kraken_op_gemm": ([i32, i32, vp, vp, vp, vp, vp, i32, i32, i32, i32, i64, i64, i64, i64,
                            vp], i32),
        "kraken_op_attention": ([i32, vp, vp, vp, i32, i32, i32, i32, i32, P(i32), i32, vp],
                                i32),
        "kraken_op_decode_attention": ([i32, vp, vp, vp, i32, i32, i32, i32, P(i32), i32, i32,
                                        i32, vp, i64, vp], i32),
        "kraken_op_decode_attention_noalloc": ([i32, vp, vp, vp, i32, i32, i32, i32, P(i32),
                                                i32, i32, i32, vp], i32),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def _check(status: int) -> None:
    if status != OK:
        raise KrakenError(status, lib().kraken_last_error().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream or None


def _cu_array(cu: Sequence[int]):
    arr = (ctypes.c_int32 * len(cu))(*[int(v) for v in cu])
    return arr


def check_device_tensor(name: str, t: torch.Tensor, dtype: torch.dtype, numel: int,
                        device: Optional[torch.device] = None) -> None:
    """Raises ValueError unless ``t`` is a contiguous GPU tensor of ``dtype`` with exactly
    ``numel`` elements (on ``device`` when given): what the C ABI's device pointers need."""
    if not getattr(t, "is_cuda", False):
        raise ValueError(f"{name} must be a GPU tensor (got {getattr(t, 'device', type(t))})")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")


def check_call_buffers(cfg: "Config", hidden: torch.Tensor, rows: int,
                       out: Optional[torch.Tensor], sub_out: Optional[torch.Tensor]) -> None:
    """Validates the buffers of a prefill / decode call of ``rows`` token rows."""
    d = cfg.d_model
    check_device_tensor("hidden", hidden, torch_dtype(dtype_code(cfg.dtype)), rows * d)
    if out is not None:
        check_device_tensor("out", out, torch.float32, rows * d, hidden.device)
    if sub_out is not None:
        check_device_tensor("sub_out", sub_out, torch.float32, cfg.n_sub * rows * d,
                            hidden.device)


def cu_from_lens(seq_lens: Sequence[int]) -> List[int]:
    cu = [0]
    for s in seq_lens:
        cu.append(cu[-1] + int(s))
    return cu


def dtype_code(dtype) -> int:
    if dtype in ("bf16", torch.bfloat16):
        return DTYPE_BF16
    if dtype in ("f16", torch.float16):
        return DTYPE_F16
    if dtype in ("f32", torch.float32):
        return DTYPE_F32
    raise ValueError(f"unsupported dtype {dtype!r}")


def torch_dtype(code: int) -> torch.dtype:
    return {DTYPE_BF16: torch.bfloat16, DTYPE_F16: torch.float16, DTYPE_F32: torch.float32}[code]


def compute_code(cfg: "Config") -> int:
    """dtype code of the MFMA operand type (the element type of a KV cache)."""
    return dtype_code(cfg.dtype if cfg.compute == "storage" else cfg.compute)


@dataclasses.dataclass
class Config:
    n_sub: int
    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int = 0
    max_tokens: int = 1
    dtype: str = "bf16"          # storage type of the weight blob and the input
    compute: str = "storage"     # MFMA operand type: "storage", "f32", "bf16" or "f16"
    ln_eps: float = 0.0
    n_kv_heads: int = 0          # key/value heads (0: n_heads; fewer: grouped-query)
    arch: str = "kraken"         # "kraken", "gpt" (standard layer) or "parallel"
    head_dim: int = 0            # 0: d_model / n_heads
    vocab: int = 0               # token embedding rows (0: no embeddings)
    max_positions: int = 0       # position embedding rows

    @property
    def kv_heads(self) -> int:
        return self.n_kv_heads or self.n_heads

    @property
    def hd(self) -> int:
        return self.head_dim or self.d_model // self.n_heads

    @property
    def stored_head_dim(self) -> int:
        """Head size as stored (32, 64 or 128): the KV cache's row length."""
        return 32 if self.hd <= 32 else 64 if self.hd <= 64 else 128

    def c_struct(self) -> _Config:
        return _Config(self.n_sub, self.n_layers, self.d_model, self.n_heads, self.d_ff,
                       self.max_tokens, dtype_code(self.dtype), COMPUTE_CODES[self.compute],
                       self.ln_eps, self.n_kv_heads, ARCH_CODES[self.arch], self.head_dim,
                       self.vocab, self.max_positions)


def weight_blob_elems(cfg: Config) -> int:
    c = cfg.c_struct()
    return int(lib().kraken_weight_blob_elems(ctypes.byref(c)))


def class_flops(cfg: Config, kernel_class: int, cu: Sequence[int]) -> float:
    c = cfg.c_struct()
    return float(lib().kraken_class_flops(ctypes.byref(c), kernel_class, _cu_array(cu),
                                          len(cu) - 1))


def pack_weights(layers: Iterable[Sequence[Mapping[str, torch.Tensor]]],
                 w_concat: Optional[torch.Tensor], cfg: Config, device=None,
                 embeddings: Optional[Mapping[str, torch.Tensor]] = None) -> torch.Tensor:
    """Flattens per-(layer, sub-layer) tensors into the blob order of kraken_load_weights:
    the layers, W_concat (Kraken only; None otherwise), then the embeddings (tok_emb,
    pos_emb, lnf_g, lnf_b) when the model has a vocabulary."""
    dt = torch_dtype(dtype_code(cfg.dtype))
    if device is None:
        device = w_concat.device if w_concat is not None else "cuda"
    blob = torch.empty(weight_blob_elems(cfg), dtype=dt, device=device)
    names = [n for n in BLOB_ORDER if cfg.arch != "parallel" or n not in ("ln2_g", "ln2_b")]
    off = 0

    def put(t):
        nonlocal off
        t = t.reshape(-1)
        blob[off:off + t.numel()].copy_(t)
        off += t.numel()

    for layer in layers:
        for sub in layer:
            for name in names:
                put(sub[name])
    if cfg.arch == "kraken":
        put(w_concat)
    elif w_concat is not None:
        raise ValueError("only the Kraken architecture has W_concat")
    if cfg.vocab:
        for name in EMB_ORDER:
            put(embeddings[name])
    if off != blob.numel():
        raise ValueError(f"blob has {off} elements, expected {blob.numel()}")
    return blob


@dataclasses.dataclass
class KVCache:
    """Device memory of a KV cache (kraken.h layout
    [L][N][2][max_seqs][heads][capacity][hd], compute type)."""
    buf: torch.Tensor
    max_seqs: int
    capacity: int

    def view(self, cfg: "Config") -> torch.Tensor:
        """The cache as a tensor [L, N, 2, max_seqs, kv_heads, capacity, hd]."""
        hd = cfg.stored_head_dim
        dt = torch_dtype(compute_code(cfg))
        return self.buf.view(dt).view(cfg.n_layers, cfg.n_sub, 2, self.max_seqs, cfg.kv_heads,
                                      self.capacity, hd)


class Kraken:
    """A Kraken model on the current HIP device (owns its device memory)."""

    def __init__(self, cfg: Config):
        self.cfg = cfg
        self._c = cfg.c_struct()
        h = ctypes.c_void_p()
        _check(lib().kraken_create(ctypes.byref(self._c), ctypes.byref(h)))
        self._h = h
        self.dtype = torch_dtype(self._c.dtype)

    @property
    def handle(self) -> ctypes.c_void_p:
        return self._h

    def close(self) -> None:
        if getattr(self, "_h", None) and self._h.value:
            lib().kraken_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def blob_elems(self) -> int:
        return int(lib().kraken_weight_blob_elems(ctypes.byref(self._c)))

    def load_weights(self, blob: torch.Tensor, stream=None) -> None:
        if blob.dtype != self.dtype or not blob.is_contiguous():
            raise ValueError("blob must be a contiguous tensor of the model dtype")
        is_dev = 1 if blob.is_cuda else 0
        _check(lib().kraken_load_weights(self._h, blob.data_ptr(),
                                         blob.numel() * blob.element_size(), is_dev,
                                         _stream(stream)))

    def prefill(self, hidden: torch.Tensor, cu_seqlens: Sequence[int],
                out: Optional[torch.Tensor] = None, sub_out=False,
                stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
        """Runs the prefill; returns (out [T, d] fp32, sub_out [N, T, d] fp32 or None)."""
        T = int(cu_seqlens[-1])
        out, sub_out = self._outputs(hidden, T, out, sub_out)
        cu = _cu_array(cu_seqlens)
        _check(lib().kraken_prefill(self._h, hidden.data_ptr(), cu, len(cu_seqlens) - 1,
                                    out.data_ptr(), _ptr(sub_out), _stream(stream)))
        return out, sub_out

    def forward_tokens(self, token_ids: Sequence[int], cu_seqlens: Sequence[int],
                       logits: Optional[torch.Tensor] = None, hidden_out=False, device=None,
                       stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
        """The whole model on packed token sequences: returns (logits [num_seqs, vocab] of
        each sequence's last token, hidden [T, d] (the unembedding's input) or None)."""
        import numpy as np
        ids = np.ascontiguousarray(np.asarray(token_ids, dtype=np.int32))
        T, B, V = int(cu_seqlens[-1]), len(cu_seqlens) - 1, self.cfg.vocab
        if ids.shape != (T,):
            raise ValueError(f"token_ids has shape {ids.shape}, expected ({T},)")
        device = device or "cuda"
        if logits is None:
            logits = torch.empty((B, V), dtype=torch.float32, device=device)
        check_device_tensor("logits", logits, torch.float32, B * V)
        if hidden_out is True:
            hidden_out = torch.empty((T, self.cfg.d_model), dtype=torch.float32,
                                     device=logits.device)
        elif hidden_out is False:
            hidden_out = None
        if hidden_out is not None:
            check_device_tensor("hidden_out", hidden_out, torch.float32, T * self.cfg.d_model,
                                logits.device)
        cu = _cu_array(cu_seqlens)
        _check(lib().kraken_forward_tokens(
            self._h, ids.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), cu, B,
            logits.data_ptr(), _ptr(hidden_out), _stream(stream)))
        return logits, hidden_out

    # ---- KV cache and decode
    def kv_cache_bytes(self, max_seqs: int, capacity: int) -> int:
        return int(lib().kraken_kv_cache_bytes(ctypes.byref(self._c), max_seqs, capacity))

    def new_kv_cache(self, max_seqs: int, capacity: int, device=None) -> "KVCache":
        """Allocates (uninitialised) device memory for a cache of max_seqs slots."""
        nbytes = self.kv_cache_bytes(max_seqs, capacity)
        if nbytes == 0:
            raise ValueError("invalid max_seqs or capacity")
        buf = torch.empty(nbytes, dtype=torch.uint8, device=device or "cuda")
        return KVCache(buf, max_seqs, capacity)

    def prefill_kv(self, hidden: torch.Tensor, cu_seqlens: Sequence[int], cache: "KVCache",
                   out: Optional[torch.Tensor] = None, sub_out=False,
                   stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
        """prefill() that also writes sequence b's keys and values into slot b of cache."""
        T = int(cu_seqlens[-1])
        out, sub_out = self._outputs(hidden, T, out, sub_out)
        self._check_cache(cache, hidden)
        cu = _cu_array(cu_seqlens)
        _check(lib().kraken_prefill_kv(self._h, hidden.data_ptr(), cu, len(cu_seqlens) - 1,
                                       out.data_ptr(), _ptr(sub_out), cache.buf.data_ptr(),
                                       cache.max_seqs, cache.capacity, _stream(stream)))
        return out, sub_out

    def decode(self, hidden: torch.Tensor, lens: Sequence[int], cache: "KVCache",
               out: Optional[torch.Tensor] = None, sub_out=False,
               stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
        """One decode step: hidden [B, d] holds one new token per sequence; lens[b] is the
        number of tokens slot b already holds.  Returns (out [B, d], sub_out [N, B, d])
        fp32; the caller advances lens by one."""
        B = len(lens)
        out, sub_out = self._outputs(hidden, B, out, sub_out)
        self._check_cache(cache, hidden)
        arr = (ctypes.c_int32 * B)(*[int(v) for v in lens])
        _check(lib().kraken_decode(self._h, hidden.data_ptr(), arr, B, out.data_ptr(),
                                   _ptr(sub_out), cache.buf.data_ptr(), cache.max_seqs,
                                   cache.capacity, _stream(stream)))
        return out, sub_out

    def _outputs(self, hidden, T, out, sub_out):
        """Allocates the outputs that are not given and validates every buffer (a contiguous
        GPU tensor of the right dtype and size), so that no host pointer, short buffer or
        wrong element type reaches the kernels."""
        d = self.cfg.d_model
        if out is None:
            out = torch.empty((T, d), dtype=torch.float32, device=hidden.device)
        if sub_out is True:
            sub_out = torch.empty((self.cfg.n_sub, T, d), dtype=torch.float32,
                                  device=hidden.device)
        elif sub_out is False:
            sub_out = None
        check_call_buffers(self.cfg, hidden, T, out, sub_out)
        return out, sub_out

    def _check_cache(self, cache: "KVCache", hidden: torch.Tensor) -> None:
        need = self.kv_cache_bytes(cache.max_seqs, cache.capacity)
        if need == 0:
            raise ValueError("invalid cache max_seqs or capacity")
        buf = cache.buf
        if not buf.is_cuda or buf.device != hidden.device or not buf.is_contiguous():
            raise ValueError("the cache must be a contiguous GPU tensor on the input's device")
        if buf.numel() * buf.element_size() < need:
            raise ValueError(f"the cache holds {buf.numel() * buf.element_size()} bytes, "
                             f"{need} needed")

    # ---- overflow check and test support
    def sync(self, stream=None) -> None:
        """Waits for the stream; raises KrakenError(ERR_OVERFLOW) if an activation exceeded
        the fp16 operand range in a call since the last sync (kraken_sync)."""
        _check(lib().kraken_sync(self._h, _stream(stream)))

    def poison_workspace(self, stream=None) -> None:
        """Fills the model's activation workspace with NaN bytes (test support)."""
        _check(lib().kraken_debug_poison_workspace(self._h, _stream(stream)))

    # ---- per-kernel timing
    def profile_enable(self, on: bool = True) -> None:
        _check(lib().kraken_profile_enable(self._h, 1 if on else 0))

    def profile_reset(self) -> None:
        _check(lib().kraken_profile_reset(self._h))

    def profile_read(self) -> dict:
        res = {}
        for k in range(K_COUNT):
            ms, n = ctypes.c_double(), ctypes.c_int64()
            _check(lib().kraken_profile_read(self._h, k, ctypes.byref(ms), ctypes.byref(n)))
            res[KERNEL_CLASS_NAMES[k]] = (ms.value, n.value)
        return res


# ----------------------------------------------------------------------------- single ops

def op_layernorm(x: torch.Tensor, x_batch_stride: int, gamma: torch.Tensor, beta: torch.Tensor,
                 out: torch.Tensor, n: int, T: int, d: int, eps: float = 1e-5,
                 stream=None) -> torch.Tensor:
    _check(lib().kraken_op_layernorm(dtype_code(out.dtype), x.data_ptr(), x_batch_stride,
                                     gamma.data_ptr(), beta.data_ptr(), out.data_ptr(), n, T, d,
                                     eps, _stream(stream)))
    return out


def op_combine_ln2(x: Optional[torch.Tensor], shared: Optional[torch.Tensor], h: torch.Tensor,
                   gamma: torch.Tensor, beta: torch.Tensor, out: torch.Tensor, n: int, T: int,
                   d: int, eps: float = 1e-5, stream=None) -> torch.Tensor:
    _check(lib().kraken_op_combine_ln2(dtype_code(out.dtype), _ptr(x), _ptr(shared),
                                       h.data_ptr(), gamma.data_ptr(), beta.data_ptr(),
                                       out.data_ptr(), n, T, d, eps, _stream(stream)))
    return out


def op_gemm(epilogue: int, A: torch.Tensor, B: torch.Tensor, C: torch.Tensor,
            bias: Optional[torch.Tensor], R: Optional[torch.Tensor], M: int, N: int, K: int,
            batch: int, sA: int, sB: int, sC: int, sR: int = 0, stream=None) -> torch.Tensor:
    _check(lib().kraken_op_gemm(dtype_code(A.dtype), epilogue, A.data_ptr(), B.data_ptr(),
                                C.data_ptr(), _ptr(bias), _ptr(R), M, N, K, batch, sA, sB, sC,
                                sR, _stream(stream)))
    return C


def vt_ld(T: int) -> int:
    return (T + 63) // 64 * 64


def op_attention(qk: torch.Tensor, vt: torch.Tensor, out: torch.Tensor, n: int, d: int,
                 n_heads: int, cu_seqlens: Sequence[int], stream=None,
                 n_kv_heads: int = 0, q_prescaled: bool = False) -> torch.Tensor:
    """Causal attention of packed sequences.  q_prescaled: the Q columns already carry
    log2(e) / sqrt(hd) (the form the prefill's Q projection produces)."""
    cu = _cu_array(cu_seqlens)
    _check(lib().kraken_op_attention(dtype_code(qk.dtype), qk.data_ptr(), vt.data_ptr(),
                                     out.data_ptr(), n, d, n_heads, n_kv_heads,
                                     1 if q_prescaled else 0, cu, len(cu_seqlens) - 1,
                                     _stream(stream)))
    return out


def op_decode_attention(qk: torch.Tensor, kv_layer: torch.Tensor, out: torch.Tensor, n: int,
                        d: int, n_heads: int, lens: Sequence[int], max_seqs: int, capacity: int,
                        work: torch.Tensor, stream=None, n_kv_heads: int = 0) -> None:
    """Attention of one new token per sequence over one layer of a KV cache."""
    B = len(lens)
    arr = (ctypes.c_int32 * B)(*[int(v) for v in lens])
    if work.dtype != torch.float32:
        raise ValueError("work must be float32")
    _check(lib().kraken_op_decode_attention(dtype_code(qk.dtype), qk.data_ptr(),
                                            kv_layer.data_ptr(), out.data_ptr(), n, d, n_heads,
                                            n_kv_heads, arr, B, max_seqs, capacity,
                                            work.data_ptr(),
                                            work.numel(), _stream(stream)))


def op_decode_attention_noalloc(qk: torch.Tensor, kv_layer: torch.Tensor, out: torch.Tensor,
                                n: int, d: int, n_heads: int, lens: Sequence[int],
                                max_seqs: int, capacity: int, stream=None,
                                n_kv_heads: int = 0) -> None:
    """op_decode_attention with the library's static scratch instead of a work buffer: the
    call allocates nothing (kraken_op_decode_attention_noalloc)."""
    B = len(lens)
    arr = (ctypes.c_int32 * B)(*[int(v) for v in lens])
    _check(lib().kraken_op_decode_attention_noalloc(dtype_code(qk.dtype), qk.data_ptr(),
                                                    kv_layer.data_ptr(), out.data_ptr(), n, d,
                                                    n_heads, n_kv_heads, arr, B, max_seqs,
                                                    capacity, _stream(stream)))
