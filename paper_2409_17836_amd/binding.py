"""ctypes binding of liblmgc (include/lmgc.h): argument marshalling only.

PyTorch supplies device memory (tensors) and streams; every step of the
LM-GC hot path runs in the library.  If liblmgc.so is missing the import of
this module still works, but every call raises: there is no fallback path.
"""
import ctypes
import os
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblmgc.so")

LMGC_OK = 0
ERRORS = {-1: "EINVAL", -2: "ENOMEM", -3: "EDEVICE", -4: "ESIZE", -5: "ECORRUPT",
          -6: "EUNSUPPORTED"}
NALPHA, NSYM = 17, 18          # with one separator token (A = 17 + escape)
HEADER_BYTES = 128

KINDS = ["embed", "norm", "gemm_qkv", "attn", "gemm_o", "gemm_up", "gemm_down", "gemm_head",
         "lse_cdf"]
KIND = {k: i for i, k in enumerate(KINDS)}


class LMGCError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class SerialParams(ctypes.Structure):
    _fields_ = [("bytes_per_value", ctypes.c_int32), ("bytes_per_group", ctypes.c_int32),
                ("msb_first", ctypes.c_int32), ("window", ctypes.c_int32),
                ("bos_id", ctypes.c_int32), ("pad_id", ctypes.c_int32),
                ("sep_id", ctypes.c_int32), ("hex_ids", ctypes.c_int32 * 16),
                ("sep2_id", ctypes.c_int32), ("renorm", ctypes.c_int32)]


class ModelConfig(ctypes.Structure):
    _fields_ = [("arch", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("d_ff", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("max_pos", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("norm_eps", ctypes.c_float)]


class DecoderState(ctypes.Structure):
    _fields_ = [("opaque", ctypes.c_uint64 * 8)]


_lib = None


def lib():
    """The loaded library; raises if liblmgc.so has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                           "(there is no fallback implementation)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u32, u64, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                  ctypes.c_uint32, ctypes.c_uint64, ctypes.c_size_t)
    P = ctypes.POINTER
    sig = {
        "lmgc_last_error": (ctypes.c_char_p, []),
        "lmgc_version": (ctypes.c_char_p, []),
        "lmgc_alphabet_size": (i32, [P(SerialParams)]),
        "lmgc_num_tokens": (i64, [i64, P(SerialParams)]),
        "lmgc_num_windows": (i64, [i64, P(SerialParams)]),
        "lmgc_serialize": (ctypes.c_int, [vp, i64, P(SerialParams), i64, i64, vp, vp, vp]),
        "lmgc_deserialize": (ctypes.c_int, [vp, i64, i64, P(SerialParams), vp]),
        "lmgc_keep_count": (i64, [i64, i32]),
        "lmgc_lossy_workspace": (i64, [i64]),
        "lmgc_sparsify_topk": (ctypes.c_int, [vp, i64, i64, vp, vp, sz, vp]),
        "lmgc_sparsify_topk_noalloc": (ctypes.c_int, [vp, i64, i64, vp, vp]),
        "lmgc_quantize_linear": (ctypes.c_int, [vp, i64, i32, vp, P(ctypes.c_float), vp, sz, vp]),
        "lmgc_sign_pack": (ctypes.c_int, [vp, i64, vp, vp]),
        "lmgc_model_num_tensors": (i32, [P(ModelConfig)]),
        "lmgc_model_tensor_info": (ctypes.c_int, [P(ModelConfig), i32, ctypes.c_char_p, sz,
                                                  P(i32), P(i64)]),
        "lmgc_model_create": (ctypes.c_int, [P(ModelConfig), P(vp), vp, P(vp)]),
        "lmgc_model_destroy": (None, [vp]),
        "lmgc_probs_workspace": (sz, [vp, i32, i32]),
        "lmgc_probs": (ctypes.c_int, [vp, vp, i32, i32, P(SerialParams), u32, vp, vp, vp, sz, vp]),
        "lmgc_step_workspace": (sz, [vp, i32, i32]),
        "lmgc_probs_stepwise": (ctypes.c_int, [vp, vp, i32, i32, P(SerialParams), u32, vp, vp, vp, sz,
                                               vp]),
        "lmgc_encode_bound": (sz, [i32, i32]),
        "lmgc_encode": (ctypes.c_int, [vp, i32, vp, vp, i32, i32, vp, sz, vp, P(sz), i32]),
        "lmgc_decode_init": (ctypes.c_int, [P(DecoderState), vp, u64]),
        "lmgc_decode_symbol": (ctypes.c_int, [P(DecoderState), vp, i32, P(i32)]),
        "lmgc_container_bound": (sz, [i64, P(SerialParams)]),
        "lmgc_codec_workspace": (sz, [vp, i64, P(SerialParams), i32]),
        "lmgc_compress": (ctypes.c_int, [vp, vp, i64, P(SerialParams), u32, i32, u64, i64, i64,
                                         vp, sz, vp, sz, P(sz), vp]),
        "lmgc_decode": (ctypes.c_int, [vp, vp, sz, i32, u64, vp, sz, vp, vp]),
        "lmgc_container_info": (ctypes.c_int, [vp, sz, P(i64), P(i32), P(i64), P(u64)]),
        "lmgc_op_gemm_bf16": (ctypes.c_int, [vp, vp, vp, i32, i32, i32, vp]),
        "lmgc_op_gemm_bf16_blocked": (ctypes.c_int, [vp, vp, vp, i32, i32, i32, i32, vp]),
        "lmgc_op_block_weights": (ctypes.c_int, [vp, vp, i32, i32, vp]),
        "lmgc_op_attention_bf16": (ctypes.c_int, [vp, vp, vp, vp, i32, i32, i32, i32, i32, vp]),
        "lmgc_timing_enable": (ctypes.c_int, [i32]),
        "lmgc_timing_kinds": (ctypes.c_int, [u32]),
        "lmgc_timing_read": (ctypes.c_int, [i32, P(ctypes.c_double), P(i64)]),
        "lmgc_probs_flops": (ctypes.c_double, [vp, i32, i32, i32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def exported_symbols() -> List[str]:
    return [n for n in dir(lib()) if n.startswith("lmgc_")]


def _check(rc: int):
    if rc != LMGC_OK:
        raise LMGCError(rc, lib().lmgc_last_error().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


# ------------------------------------------------------------ conversions --
def serial_params(spec) -> SerialParams:
    """From any object with the SerialParams field names (e.g. synth.SerialSpec)."""
    p = SerialParams()
    for f, _ in SerialParams._fields_:
        if f == "hex_ids":
            ids = list(spec.hex_ids)
            assert len(ids) == 16
            p.hex_ids = (ctypes.c_int32 * 16)(*ids)
        elif f == "sep2_id":
            p.sep2_id = int(getattr(spec, "sep2_id", -1))
        elif f == "renorm":
            p.renorm = int(getattr(spec, "renorm", 0))
        else:
            setattr(p, f, int(getattr(spec, f)))
    return p


def alphabet_size(sp: SerialParams) -> int:
    """Coded alphabet size A (17, or 18 with a second separator token)."""
    n = int(lib().lmgc_alphabet_size(ctypes.byref(sp)))
    if n < 0:
        raise LMGCError(-1, lib().lmgc_last_error().decode())
    return n


def model_config(shape) -> ModelConfig:
    """From any object with ModelShape fields (arch "llama"/"gpt2", dtype "f32"/"bf16")."""
    c = ModelConfig()
    c.arch = {"llama": 0, "gpt2": 1}[shape.arch]
    c.dtype = {"f32": 0, "bf16": 1}[shape.dtype]
    for f in ("n_layers", "d_model", "n_heads", "n_kv_heads", "d_ff", "vocab", "max_pos"):
        setattr(c, f, int(getattr(shape, f)))
    c.rope_theta = float(shape.rope_theta)
    c.norm_eps = float(shape.norm_eps)
    return c


# ---------------------------------------------------------- serialisation --
def num_tokens(n_values: int, sp: SerialParams) -> int:
    return int(lib().lmgc_num_tokens(n_values, ctypes.byref(sp)))


def num_windows(n_values: int, sp: SerialParams) -> int:
    return int(lib().lmgc_num_windows(n_values, ctypes.byref(sp)))


def serialize(values, sp: SerialParams, first_window: int = 0, n_windows: int = None,
              tokens=None, sym=None, want_sym: bool = True, stream=None):
    """values: 1-D CUDA tensor (float32 / uint8 / int16) -> (tokens [nw, W] int32, sym [nw, W] uint8)."""
    import torch
    n = values.numel()
    assert values.element_size() == sp.bytes_per_value and values.is_contiguous()
    if n_windows is None:
        n_windows = num_windows(n, sp) - first_window
    W = sp.window
    if tokens is None:
        tokens = torch.empty((n_windows, W), dtype=torch.int32, device=values.device)
    if sym is None and want_sym:
        sym = torch.empty((n_windows, W), dtype=torch.uint8, device=values.device)
    _check(lib().lmgc_serialize(_ptr(values), n, ctypes.byref(sp), first_window, n_windows,
                                _ptr(tokens), _ptr(sym), _stream(stream)))
    return tokens, sym


def deserialize(sym: np.ndarray, n_values: int, sp: SerialParams, dtype) -> np.ndarray:
    s = np.ascontiguousarray(sym, dtype=np.uint8)
    out = np.empty(n_values * sp.bytes_per_value, np.uint8)
    _check(lib().lmgc_deserialize(s.ctypes.data, s.size, n_values, ctypes.byref(sp),
                                  out.ctypes.data))
    return out.view(dtype)


# ------------------------------------------------------------ lossy steps --
def keep_count(n_values: int, percent: int) -> int:
    """Values sparsification keeps at `percent` percent (Sec. 5.4)."""
    k = int(lib().lmgc_keep_count(n_values, percent))
    if k < 0:
        _check(k)
    return k


def lossy_workspace(n_values: int) -> int:
    n = int(lib().lmgc_lossy_workspace(n_values))
    if n < 0:
        _check(n)
    return n


def sparsify_topk(values, k: int, out=None, ws=None, stream=None):
    """Keep the k largest-magnitude values of a CUDA float32 vector (Sec. 5.4);
    out may be values itself."""
    import torch
    assert values.dtype == torch.float32 and values.is_contiguous()
    n = values.numel()
    if out is None:
        out = torch.empty_like(values)
    if ws is None:
        ws = workspace(lossy_workspace(n), values.device)
    _check(lib().lmgc_sparsify_topk(_ptr(values), n, int(k), _ptr(out), _ptr(ws), ws.numel(),
                                    _stream(stream)))
    return out


def sparsify_topk_noalloc(values, k: int, out, stream=None):
    """sparsify_topk on the library's own device scratch: no workspace, and
    the call allocates nothing (out must be given; it may be values)."""
    import torch
    assert values.dtype == torch.float32 and values.is_contiguous()
    assert out.dtype == torch.float32 and out.numel() == values.numel()
    _check(lib().lmgc_sparsify_topk_noalloc(_ptr(values), values.numel(), int(k), _ptr(out),
                                            _stream(stream)))
    return out


def quantize_linear(values, bits: int, out=None, ws=None, stream=None):
    """Eq. 4 indices of a CUDA float32 vector -> (indices, min, max).  Indices
    are uint8 for bits <= 8, else int16 storage holding uint16 values."""
    import torch
    assert values.dtype == torch.float32 and values.is_contiguous()
    n = values.numel()
    if out is None:
        out = torch.empty(n, dtype=torch.uint8 if bits <= 8 else torch.int16, device=values.device)
    if ws is None:
        ws = workspace(lossy_workspace(n), values.device)
    mm = (ctypes.c_float * 2)()
    _check(lib().lmgc_quantize_linear(_ptr(values), n, int(bits), _ptr(out), mm, _ptr(ws), ws.numel(),
                                      _stream(stream)))
    return out, float(mm[0]), float(mm[1])


def sign_pack(values, out=None, stream=None):
    """SignSGD bits of a CUDA float32 vector, eight per byte, first value in bit 7."""
    import torch
    assert values.dtype == torch.float32 and values.is_contiguous()
    n = values.numel()
    if out is None:
        out = torch.empty((n + 7) // 8, dtype=torch.uint8, device=values.device)
    _check(lib().lmgc_sign_pack(_ptr(values), n, _ptr(out), _stream(stream)))
    return out


def lossy_prepare(values, steps, stream=None):
    """Apply lossy steps [(kind, arg)] left to right on the GPU: ("sparsify",
    percent), ("quantize", bits), ("sign", 0).  Returns the value stream."""
    x = values
    ws = None
    for kind, arg in steps:
        if kind == "sparsify":
            if ws is None:
                ws = workspace(lossy_workspace(x.numel()), x.device)
            x = sparsify_topk(x, keep_count(x.numel(), int(arg)), ws=ws, stream=stream)
        elif kind == "quantize":
            if ws is None:
                ws = workspace(lossy_workspace(x.numel()), x.device)
            x = quantize_linear(x, int(arg), ws=ws, stream=stream)[0]
        elif kind == "sign":
            x = sign_pack(x, stream=stream)
        else:
            raise ValueError(f"unknown lossy step {kind!r}")
    return x


# ------------------------------------------------------------------ model --
def manifest(cfg: ModelConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    L = lib()
    n = L.lmgc_model_num_tensors(ctypes.byref(cfg))
    if n < 0:
        _check(-1)
    out = []
    name = ctypes.create_string_buffer(128)
    nd = ctypes.c_int32()
    shape = (ctypes.c_int64 * 2)()
    for i in range(n):
        _check(L.lmgc_model_tensor_info(ctypes.byref(cfg), i, name, 128, ctypes.byref(nd), shape))
        out.append((name.value.decode(), tuple(shape[:nd.value])))
    return out


class Model:
    """A decoder on the GPU.  weights: CUDA tensors in manifest order (bf16
    models: torch.bfloat16 or int16/uint16 bit patterns; f32: float32)."""

    def __init__(self, cfg: ModelConfig, weights: Sequence, stream=None):
        man = manifest(cfg)
        assert len(weights) == len(man), (len(weights), len(man))
        for (name, shape), w in zip(man, weights):
            assert tuple(w.shape) == tuple(shape), (name, tuple(w.shape), shape)
            assert w.is_contiguous()
        arr = (ctypes.c_void_p * len(man))(*[_ptr(w) for w in weights])
        h = ctypes.c_void_p()
        _check(lib().lmgc_model_create(ctypes.byref(cfg), arr, _stream(stream), ctypes.byref(h)))
        self.cfg = cfg
        self.handle = h

    def close(self):
        if self.handle:
            lib().lmgc_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def probs_workspace(self, B: int, W: int) -> int:
        return int(lib().lmgc_probs_workspace(self.handle, B, W))

    def step_workspace(self, B: int, W: int) -> int:
        return int(lib().lmgc_step_workspace(self.handle, B, W))

    def codec_workspace(self, n_values: int, sp: SerialParams, batch: int) -> int:
        return int(lib().lmgc_codec_workspace(self.handle, n_values, ctypes.byref(sp), batch))

    def flops(self, B: int, W: int, kind: str) -> float:
        return float(lib().lmgc_probs_flops(self.handle, B, W, KIND[kind]))


def workspace(nbytes: int, device="cuda"):
    import torch
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def probs(model: Model, tokens, sp: SerialParams, total: int = 1 << 16, want_logp: bool = True,
          ws=None, cdf=None, logp=None, stream=None):
    """tokens: CUDA int32 [B, W] -> (cdf int32 [B, W, A + 2] holding uint32 values,
    logp float32 [B, W, A]) with A = alphabet_size(sp)."""
    import torch
    B, W = tokens.shape
    assert tokens.dtype == torch.int32 and tokens.is_contiguous()
    na = alphabet_size(sp)
    need = model.probs_workspace(B, W)
    if ws is None:
        ws = workspace(need, tokens.device)
    if cdf is None:
        cdf = torch.empty((B, W, na + 2), dtype=torch.int32, device=tokens.device)
    if logp is None and want_logp:
        logp = torch.empty((B, W, na), dtype=torch.float32, device=tokens.device)
    _check(lib().lmgc_probs(model.handle, _ptr(tokens), B, W, ctypes.byref(sp), total, _ptr(cdf),
                            _ptr(logp), _ptr(ws), ws.numel(), _stream(stream)))
    return cdf, logp


def probs_stepwise(model: Model, tokens, sp: SerialParams, total: int = 1 << 16,
                   want_logp: bool = True, ws=None, stream=None):
    """lmgc_probs_stepwise: the same outputs as probs(), computed position by
    position through the K/V cache (the decoder's path); B <= 32."""
    import torch
    B, W = tokens.shape
    assert tokens.dtype == torch.int32 and tokens.is_contiguous()
    na = alphabet_size(sp)
    if ws is None:
        ws = workspace(model.step_workspace(B, W), tokens.device)
    cdf = torch.empty((B, W, na + 2), dtype=torch.int32, device=tokens.device)
    logp = torch.empty((B, W, na), dtype=torch.float32, device=tokens.device) if want_logp else None
    _check(lib().lmgc_probs_stepwise(model.handle, _ptr(tokens), B, W, ctypes.byref(sp), total,
                                     _ptr(cdf), _ptr(logp), _ptr(ws), ws.numel(), _stream(stream)))
    return cdf, logp


# ------------------------------------------------------------------ coder --
def encode(cdf: np.ndarray, sym: np.ndarray, lens: np.ndarray, n_threads: int = 0):
    """cdf [n_win, W, nsym+1] uint32, sym [n_win, W] uint8, lens [n_win] -> (payloads bytes, bits uint32[n_win])."""
    cdf = np.ascontiguousarray(cdf, dtype=np.uint32)
    sym = np.ascontiguousarray(sym, dtype=np.uint8)
    lens = np.ascontiguousarray(lens, dtype=np.int32)
    n_win, W = sym.shape
    nsym = cdf.shape[-1] - 1
    cap = int(lib().lmgc_encode_bound(n_win, W))
    out = np.empty(max(cap, 1), np.uint8)
    bits = np.zeros(n_win, np.uint32)
    used = ctypes.c_size_t()
    _check(lib().lmgc_encode(cdf.ctypes.data, nsym, sym.ctypes.data, lens.ctypes.data, n_win, W,
                             out.ctypes.data, cap, bits.ctypes.data, ctypes.byref(used), n_threads))
    return out[:used.value].tobytes(), bits


class StepDecoder:
    def __init__(self, payload: bytes, nbits: int):
        self._buf = np.frombuffer(payload, np.uint8).copy() if len(payload) else np.zeros(1, np.uint8)
        self._st = DecoderState()
        _check(lib().lmgc_decode_init(ctypes.byref(self._st), self._buf.ctypes.data, nbits))

    def decode(self, cdf_row: np.ndarray) -> int:
        row = np.ascontiguousarray(cdf_row, dtype=np.uint32)
        out = ctypes.c_int32()
        _check(lib().lmgc_decode_symbol(ctypes.byref(self._st), row.ctypes.data, row.size - 1,
                                        ctypes.byref(out)))
        return out.value


# ------------------------------------------------------------------ codec --
def compress(model: Model, values, sp: SerialParams, total: int = 1 << 16, batch: int = 8,
             model_tag: int = 0, first_window: int = 0, n_windows: int = -1, ws=None,
             stream=None) -> bytes:
    n = values.numel()
    nw = num_windows(n, sp)
    cnt = (nw - first_window) if n_windows < 0 else n_windows
    cap = 128 + 4 * cnt + int(lib().lmgc_encode_bound(max(cnt, 1), sp.window))
    out = np.empty(cap, np.uint8)
    if ws is None:
        ws = workspace(model.codec_workspace(n, sp, batch), values.device)
    used = ctypes.c_size_t()
    _check(lib().lmgc_compress(model.handle, _ptr(values), n, ctypes.byref(sp), total, batch,
                               model_tag, first_window, n_windows, _ptr(ws), ws.numel(),
                               out.ctypes.data, cap, ctypes.byref(used), _stream(stream)))
    return out[:used.value].tobytes()


def container_info(buf: bytes):
    a = np.frombuffer(buf, np.uint8)
    nv, bpv, nw, tag = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int64(), ctypes.c_uint64()
    _check(lib().lmgc_container_info(a.ctypes.data, a.size, ctypes.byref(nv), ctypes.byref(bpv),
                                     ctypes.byref(nw), ctypes.byref(tag)))
    return dict(n_values=nv.value, bytes_per_value=bpv.value, n_windows=nw.value,
                model_tag=tag.value)


def decode(model: Model, buf: bytes, batch: int = 8, model_tag: int = 0, ws=None,
           stream=None, dtype=np.float32) -> np.ndarray:
    info = container_info(buf)
    a = np.frombuffer(buf, np.uint8).copy()
    out = np.empty(info["n_values"] * info["bytes_per_value"], np.uint8)
    W = int.from_bytes(buf[28:32], "little")
    sp = SerialParams()
    sp.window = W
    if ws is None:
        ws = workspace(model.codec_workspace(info["n_values"], sp, batch))
    _check(lib().lmgc_decode(model.handle, a.ctypes.data, a.size, batch, model_tag, _ptr(ws),
                             ws.numel(), out.ctypes.data, _stream(stream)))
    return out.view(dtype)


# ----------------------------------------------------------- kernel level --
def op_gemm_bf16(a, b, c=None, stream=None):
    """a [M, K], b [N, K] bf16 CUDA tensors -> c [M, N] float32 = a b^T."""
    import torch
    M, K = a.shape
    N = b.shape[0]
    if c is None:
        c = torch.empty((M, N), dtype=torch.float32, device=a.device)
    _check(lib().lmgc_op_gemm_bf16(_ptr(a), _ptr(b), _ptr(c), M, N, K, _stream(stream)))
    return c


OP_KINDS = {"store": 0, "resid": 1, "swiglu": 2}


def op_block_weights(b, stream=None):
    """b [N, K] bf16 CUDA tensor (row-major) -> the same matrix in MFMA blocks."""
    import torch
    N, K = b.shape
    out = torch.empty_like(b)
    _check(lib().lmgc_op_block_weights(_ptr(b), _ptr(out), N, K, _stream(stream)))
    return out


def op_gemm_bf16_blocked(a, b_blocked, kind: str, out=None, stream=None):
    """The model's blocked-weight product with its epilogue: "store" (float32
    [M, N] = a b^T), "resid" (out += a b^T; out given), "swiglu" (bf16
    [M, N/2], b's rows gate/up interleaved in groups of 32)."""
    import torch
    M, K = a.shape
    N = b_blocked.shape[0]
    if out is None:
        out = (torch.empty((M, N // 2), dtype=torch.bfloat16, device=a.device) if kind == "swiglu"
               else torch.zeros((M, N), dtype=torch.float32, device=a.device))
    _check(lib().lmgc_op_gemm_bf16_blocked(_ptr(a), _ptr(b_blocked), _ptr(out), M, N, K, OP_KINDS[kind],
                                           _stream(stream)))
    return out


def op_attention_bf16(q, k, vt, o=None, stream=None):
    """q [B, Hq, W, hd], k [B, Hkv, W, hd], vt = V transposed [B, Hkv, hd, W],
    all bf16 -> o [B*W, Hq*hd] bf16."""
    import torch
    B, Hq, W, hd = q.shape
    Hkv = k.shape[1]
    if o is None:
        o = torch.empty((B * W, Hq * hd), dtype=torch.bfloat16, device=q.device)
    _check(lib().lmgc_op_attention_bf16(_ptr(q), _ptr(k), _ptr(vt), _ptr(o), B, Hq, Hkv, W, hd,
                                        _stream(stream)))
    return o


# ----------------------------------------------------------------- timing --
def timing_enable(on: bool = True):
    _check(lib().lmgc_timing_enable(1 if on else 0))


def timing_kinds(kinds=None):
    """lmgc_timing_kinds: record events only for these kinds (None: all)."""
    names = list(KIND) if kinds is None else list(kinds)
    mask = 0
    for k in names:
        mask |= 1 << KIND[k]
    _check(lib().lmgc_timing_kinds(mask))


def timing_read(kind: str) -> Tuple[float, int]:
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check(lib().lmgc_timing_read(KIND[kind], ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
