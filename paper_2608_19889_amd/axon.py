"""Python binding of the C ABI in ``include/axon.h`` (ctypes).

Argument marshalling only: every step of the forward pass runs in the HIP
kernels of ``libaxon.so``.  torch supplies device memory and the current
stream; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libaxon.so")

AXON_OK = 0
AXON_E_INVALID = -1
AXON_E_SHAPE = -2
AXON_E_MISSING = -3
AXON_E_DTYPE = -4
AXON_E_CAPACITY = -5
AXON_E_OOM = -6
AXON_E_HIP = -7
AXON_BF16 = 1
AXON_F32 = 2
AXON_ARCH_LLAMA = 0
AXON_ARCH_GPT2 = 1

STATUS_NAMES = {0: "AXON_OK", -1: "AXON_E_INVALID", -2: "AXON_E_SHAPE", -3: "AXON_E_MISSING",
                -4: "AXON_E_DTYPE", -5: "AXON_E_CAPACITY", -6: "AXON_E_OOM", -7: "AXON_E_HIP"}

EXPORTED = ["axon_init_model", "axon_prefill", "axon_decode_step", "axon_decode_step_noalloc", "axon_step", "axon_reset_slot", "axon_loss_and_grads",
            "axon_slot_lengths", "axon_timing_enable", "axon_timing_records", "axon_free", "axon_last_error"]

# kernel classes of the timing records
T_GEMV, T_GEMM, T_ATTN_DECODE, T_ATTN_PREFILL, T_GEMV_GROUPED, T_ATTN_BWD = 0, 1, 2, 3, 4, 5


class AxonConfig(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("intermediate", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_theta", ctypes.c_double), ("qkv_bias", ctypes.c_int32),
                ("tie_embeddings", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("max_batch", ctypes.c_int32), ("max_seq", ctypes.c_int32),
                ("max_tokens", ctypes.c_int32), ("kv_page_size", ctypes.c_int32),
                ("kv_num_pages", ctypes.c_int32), ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("moe_intermediate", ctypes.c_int32), ("n_shared_experts", ctypes.c_int32),
                ("first_moe_layer", ctypes.c_int32), ("norm_topk_prob", ctypes.c_int32),
                ("sliding_window", ctypes.c_int32), ("arch", ctypes.c_int32), ("max_positions", ctypes.c_int32)]


class AxonWeight(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 2), ("data", ctypes.c_void_p),
                ("on_device", ctypes.c_int32)]


class AxonError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


_lib = None


def lib():
    """Load ``libaxon.so``; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        L.axon_init_model.argtypes = [ctypes.POINTER(AxonConfig), ctypes.POINTER(AxonWeight), ctypes.c_int32,
                                      ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]
        L.axon_init_model.restype = ctypes.c_int
        L.axon_prefill.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                   ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_void_p]
        L.axon_prefill.restype = ctypes.c_int
        L.axon_decode_step.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p]
        L.axon_decode_step.restype = ctypes.c_int
        L.axon_decode_step_noalloc.argtypes = L.axon_decode_step.argtypes
        L.axon_decode_step_noalloc.restype = ctypes.c_int
        L.axon_step.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                ctypes.POINTER(ctypes.c_int32), ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.axon_step.restype = ctypes.c_int
        L.axon_reset_slot.argtypes = [ctypes.c_void_p, ctypes.c_int32]
        L.axon_loss_and_grads.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.POINTER(ctypes.c_int32), ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.POINTER(AxonWeight), ctypes.c_int32, ctypes.c_void_p]
        L.axon_loss_and_grads.restype = ctypes.c_int
        L.axon_reset_slot.restype = ctypes.c_int
        L.axon_slot_lengths.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32]
        L.axon_slot_lengths.restype = ctypes.c_int
        L.axon_timing_enable.argtypes = [ctypes.c_void_p, ctypes.c_int32]
        L.axon_timing_enable.restype = ctypes.c_int
        L.axon_timing_records.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                                          ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_float),
                                          ctypes.c_int32]
        L.axon_timing_records.restype = ctypes.c_int
        L.axon_free.argtypes = [ctypes.c_void_p]
        L.axon_free.restype = None
        L.axon_last_error.argtypes = []
        L.axon_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def last_error() -> str:
    return lib().axon_last_error().decode()


def _check(rc: int):
    if rc < 0:
        raise AxonError(rc, last_error())
    return rc


def make_config(shape: dict, max_batch: int, max_seq: int, max_tokens: int = 0, page_size: int = 0,
                num_pages: int = 0) -> AxonConfig:
    """``shape`` uses HF-style keys (hidden_size, num_hidden_layers, ...);
    ``model_type == "gpt2"`` selects the GPT-2 family (layer_norm_epsilon,
    max_position_embeddings)."""
    gpt2 = shape.get("model_type") == "gpt2"
    return AxonConfig(
        hidden=shape["hidden_size"], n_layers=shape["num_hidden_layers"],
        n_heads=shape["num_attention_heads"], n_kv_heads=shape["num_key_value_heads"],
        head_dim=shape["head_dim"], intermediate=shape["intermediate_size"], vocab=shape["vocab_size"],
        rms_eps=shape["layer_norm_epsilon"] if gpt2 else shape["rms_norm_eps"],
        rope_theta=0.0 if gpt2 else shape["rope_theta"],
        qkv_bias=int(bool(shape["attention_bias"])), tie_embeddings=int(bool(shape["tie_word_embeddings"])),
        dtype=AXON_BF16 if shape["dtype"] == "bf16" else AXON_F32, max_batch=max_batch, max_seq=max_seq,
        max_tokens=max_tokens, kv_page_size=page_size, kv_num_pages=num_pages,
        n_experts=int(shape.get("n_routed_experts") or 0), top_k=int(shape.get("num_experts_per_tok") or 0),
        moe_intermediate=int(shape.get("moe_intermediate_size") or 0),
        n_shared_experts=int(shape.get("n_shared_experts") or 0),
        first_moe_layer=int(shape.get("first_k_dense_replace") or 0),
        norm_topk_prob=int(bool(shape.get("norm_topk_prob"))),
        sliding_window=int(shape.get("sliding_window") or 0), arch=AXON_ARCH_GPT2 if gpt2 else AXON_ARCH_LLAMA,
        max_positions=int(shape.get("max_position_embeddings") or 0) if gpt2 else 0)


def make_weights(weights: dict) -> tuple[ctypes.Array, list]:
    """Marshal {name: tensor} into an axon_weight array; returns it together
    with the objects that must stay alive for the call."""
    keep = []
    arr = (AxonWeight * len(weights))()
    for i, (name, t) in enumerate(weights.items()):
        if not t.is_contiguous():
            t = t.contiguous()
        keep.append(t)
        nb = name.encode()
        keep.append(nb)
        arr[i].name = nb
        arr[i].dtype = AXON_BF16 if t.dtype == torch.bfloat16 else (AXON_F32 if t.dtype == torch.float32 else 0)
        arr[i].ndim = t.dim()
        arr[i].shape[0] = t.shape[0] if t.dim() >= 1 else 0
        arr[i].shape[1] = t.shape[1] if t.dim() >= 2 else 0
        arr[i].data = t.data_ptr()
        arr[i].on_device = int(t.is_cuda)
    return arr, keep


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


class Model:
    """One decoder model resident on the current GPU."""

    def __init__(self, shape: dict, weights: dict, max_batch: int, max_seq: int, max_tokens: int = 0,
                 page_size: int = 0, num_pages: int = 0, stream=None):
        self.shape = dict(shape)
        self.vocab = shape["vocab_size"]
        self.max_batch = max_batch
        self.cfg = make_config(shape, max_batch, max_seq, max_tokens, page_size, num_pages)
        arr, keep = make_weights(weights)
        handle = ctypes.c_void_p()
        _check(lib().axon_init_model(ctypes.byref(self.cfg), arr, len(weights), ctypes.c_void_p(_stream(stream)),
                                     ctypes.byref(handle)))
        del keep
        self._h = handle

    # ---- calls
    def prefill(self, tokens: torch.Tensor, cu_seqlens: list, block_table: torch.Tensor | None = None,
                all_logits: bool = False, logits: torch.Tensor | None = None,
                next_tokens: torch.Tensor | None = None, want_logits: bool = True, stream=None):
        """tokens: device int32 [sum S_b]; cu_seqlens: host list of batch+1 ints;
        block_table: host int32 [batch, stride] for a paged cache.  Returns
        (logits or None, next_tokens)."""
        dev = tokens.device
        B = len(cu_seqlens) - 1
        cu_h = (ctypes.c_int32 * (B + 1))(*[int(c) for c in cu_seqlens])
        cu_d = torch.tensor([int(c) for c in cu_seqlens], dtype=torch.int32, device=dev)
        rows = int(cu_seqlens[-1]) if all_logits else B
        if logits is None and (want_logits or all_logits):
            logits = torch.empty((rows, self.vocab), dtype=torch.float32, device=dev)
        if next_tokens is None:
            next_tokens = torch.empty((B,), dtype=torch.int32, device=dev)
        bt_ptr, stride = None, 0
        if block_table is not None:
            bt = block_table.to("cpu", torch.int32).contiguous()
            stride = bt.shape[1]
            bt_ptr = ctypes.cast(bt.data_ptr(), ctypes.POINTER(ctypes.c_int32))
        _check(lib().axon_prefill(self._h, B, tokens.data_ptr(), cu_d.data_ptr(), cu_h, bt_ptr, stride,
                                  int(all_logits), logits.data_ptr() if logits is not None else None,
                                  next_tokens.data_ptr(), ctypes.c_void_p(_stream(stream))))
        self._keep = (cu_d, tokens)
        return logits, next_tokens

    def loss_and_grads(self, tokens: torch.Tensor, cu_seqlens: list, targets: torch.Tensor, grads: dict,
                       loss: torch.Tensor | None = None, stream=None):
        """Backward pass (axon_loss_and_grads): tokens / targets device int32
        [sum S_b] (targets -1 or outside [0, V) are not counted); grads: {weight
        name: device float32 tensor of that weight's shape}, overwritten with
        the gradient of the mean cross-entropy.  Returns the loss (device
        float32 [1])."""
        dev = tokens.device
        B = len(cu_seqlens) - 1
        cu_h = (ctypes.c_int32 * (B + 1))(*[int(c) for c in cu_seqlens])
        cu_d = torch.tensor([int(c) for c in cu_seqlens], dtype=torch.int32, device=dev)
        if loss is None:
            loss = torch.empty((1,), dtype=torch.float32, device=dev)
        arr, keep = make_weights(grads)
        _check(lib().axon_loss_and_grads(self._h, B, tokens.data_ptr(), cu_d.data_ptr(), cu_h, targets.data_ptr(),
                                         loss.data_ptr(), arr, len(grads), ctypes.c_void_p(_stream(stream))))
        self._keep = (cu_d, tokens, targets, keep)
        return loss

    def decode_step(self, tokens: torch.Tensor, logits: torch.Tensor | None = None,
                    next_tokens: torch.Tensor | None = None, stream=None):
        """tokens: device int32 [batch].  Returns (logits or None, next_tokens)."""
        B = tokens.shape[0]
        if next_tokens is None:
            next_tokens = torch.empty((B,), dtype=torch.int32, device=tokens.device)
        _check(lib().axon_decode_step(self._h, B, tokens.data_ptr(),
                                      logits.data_ptr() if logits is not None else None,
                                      next_tokens.data_ptr(), ctypes.c_void_p(_stream(stream))))
        return logits, next_tokens

    def decode_step_noalloc(self, tokens: torch.Tensor, logits: torch.Tensor | None = None,
                            next_tokens: torch.Tensor = None, stream=None):
        """axon_decode_step_noalloc: the decode step with its work buffers in the
        library's fixed per-GPU array (nothing is allocated by the call; the
        caller provides ``next_tokens``, device int32 [batch]).  Returns
        (logits or None, next_tokens)."""
        if next_tokens is None:
            raise ValueError("decode_step_noalloc needs a caller-provided next_tokens buffer")
        _check(lib().axon_decode_step_noalloc(self._h, tokens.shape[0], tokens.data_ptr(),
                                              logits.data_ptr() if logits is not None else None,
                                              next_tokens.data_ptr(), ctypes.c_void_p(_stream(stream))))
        return logits, next_tokens

    def step(self, tokens: torch.Tensor, cu_seqlens: list, slots: list, fresh: list | None = None,
             block_rows: torch.Tensor | None = None, logits: torch.Tensor | None = None,
             next_tokens: torch.Tensor | None = None, want_logits: bool = True, stream=None,
             cu_device: torch.Tensor | None = None):
        """One continuous-batching step (axon_step).  tokens: device int32
        [sum n_i]; cu_seqlens: host list of n+1 ints; slots / fresh: host lists
        of n ints; block_rows: host int32 [n, stride] page rows (paged cache) or
        None; cu_device: optional device int32 buffer (>= n+1 entries) that
        receives cu_seqlens, so that its address stays fixed across calls.
        Returns (logits [n, V] or None, next_tokens [n])."""
        dev = tokens.device
        n = len(slots)
        cu_h = (ctypes.c_int32 * (n + 1))(*[int(c) for c in cu_seqlens])
        if cu_device is not None:
            cu_d = cu_device
            cu_d[:n + 1].copy_(torch.tensor([int(c) for c in cu_seqlens], dtype=torch.int32), non_blocking=True)
        else:
            cu_d = torch.tensor([int(c) for c in cu_seqlens], dtype=torch.int32, device=dev)
        sl_h = (ctypes.c_int32 * n)(*[int(x) for x in slots])
        fr_h = (ctypes.c_int32 * n)(*[int(x) for x in fresh]) if fresh is not None else None
        if logits is None and want_logits:
            logits = torch.empty((n, self.vocab), dtype=torch.float32, device=dev)
        if next_tokens is None:
            next_tokens = torch.empty((n,), dtype=torch.int32, device=dev)
        bt_ptr, stride = None, 0
        if block_rows is not None:
            bt = block_rows.to("cpu", torch.int32).contiguous()
            stride = bt.shape[1]
            bt_ptr = ctypes.cast(bt.data_ptr(), ctypes.POINTER(ctypes.c_int32))
        _check(lib().axon_step(self._h, n, sl_h, fr_h, tokens.data_ptr(), cu_d.data_ptr(), cu_h, bt_ptr, stride,
                               logits.data_ptr() if logits is not None else None, next_tokens.data_ptr(),
                               ctypes.c_void_p(_stream(stream))))
        self._keep = (cu_d, tokens)
        return logits, next_tokens

    def reset_slot(self, slot: int):
        """Evict the sequence of ``slot`` (axon_reset_slot)."""
        _check(lib().axon_reset_slot(self._h, int(slot)))

    def lengths(self) -> list[int]:
        buf = (ctypes.c_int32 * self.max_batch)()
        n = _check(lib().axon_slot_lengths(self._h, buf, self.max_batch))
        return list(buf)[:n]

    def timing(self, enable: bool):
        _check(lib().axon_timing_enable(self._h, int(enable)))

    def timing_records(self):
        """List of (kernel class, (d0, d1, d2), milliseconds)."""
        n = _check(lib().axon_timing_records(self._h, None, None, None, 0))
        cls = (ctypes.c_int32 * max(n, 1))()
        dims = (ctypes.c_int32 * max(3 * n, 1))()
        ms = (ctypes.c_float * max(n, 1))()
        _check(lib().axon_timing_records(self._h, cls, dims, ms, n))
        return [(cls[i], (dims[3 * i], dims[3 * i + 1], dims[3 * i + 2]), ms[i]) for i in range(n)]

    def close(self):
        if getattr(self, "_h", None):
            lib().axon_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def init_status(cfg: AxonConfig, weights: dict) -> tuple[int, str]:
    """Call axon_init_model and return (status, message) without raising (for
    validation tests).  A successful handle is freed immediately."""
    arr, keep = make_weights(weights)
    handle = ctypes.c_void_p()
    rc = lib().axon_init_model(ctypes.byref(cfg), arr, len(weights), None, ctypes.byref(handle))
    msg = last_error()
    if rc == AXON_OK:
        lib().axon_free(handle)
    del keep
    return rc, msg
