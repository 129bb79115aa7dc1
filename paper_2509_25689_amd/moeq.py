"""ctypes binding of the moeq C interface (include/moeq.h).

Argument marshalling only: every step of the layer runs in the HIP library
``libmoeq.so`` next to this file.  Importing fails loudly when the library has
not been built; nothing here falls back to another implementation.

The functions keep the C names.  Pointers are plain integers (device or host
addresses); streams are ``hipStream_t`` values as integers (0 = default).
``Layer`` is a small convenience wrapper that takes numpy arrays (host weights)
or torch tensors (device weights / activations) and keeps nothing but the
handle.
"""
import ctypes
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoeq.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "moeq.h")

MOEQ_OK = 0
MOEQ_ERR_INVALID_ARG = -1
MOEQ_ERR_UNSUPPORTED = -2
MOEQ_ERR_OUT_OF_MEMORY = -3
MOEQ_ERR_DEVICE = -4
MOEQ_ERR_CAPACITY = -5
STATUS_NAMES = {0: "OK", -1: "INVALID_ARG", -2: "UNSUPPORTED", -3: "OUT_OF_MEMORY",
                -4: "DEVICE", -5: "CAPACITY"}

MOEQ_PROJ_GATE, MOEQ_PROJ_UP, MOEQ_PROJ_DOWN = 0, 1, 2
MOEQ_WEIGHTS_HOST, MOEQ_WEIGHTS_DEVICE = 0, 1
MOEQ_PATH_AUTO, MOEQ_PATH_DECODE, MOEQ_PATH_PREFILL = 0, 1, 2
MOEQ_DECODER_EXACT, MOEQ_DECODER_GEMV_SUBNORMAL, MOEQ_DECODER_GEMM_F16 = 0, 1, 2


class MoeqError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        super().__init__(f"moeq {STATUS_NAMES.get(status, status)}: {message}")


class moeq_config(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("inter", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("n_shared", ctypes.c_int32),
                ("n_group", ctypes.c_int32), ("topk_group", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("group_topn", ctypes.c_int32),
                ("norm_topk", ctypes.c_int32), ("routed_scale", ctypes.c_float),
                ("max_tokens", ctypes.c_int32), ("decode_max_tokens", ctypes.c_int32),
                ("regroup", ctypes.c_int32)]


class moeq_qtensor(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("codes", ctypes.c_void_p),
                ("scales", ctypes.c_void_p)]


MOEQ_TENSOR_OTHER, MOEQ_TENSOR_ROUTED_GATE, MOEQ_TENSOR_ROUTED_UP, MOEQ_TENSOR_ROUTED_DOWN = 0, 1, 2, 3
MOEQ_PLAN_MAX_LEVELS = 8


class moeq_plan_params(ctypes.Structure):
    _fields_ = [("n_levels", ctypes.c_int32), ("width64", ctypes.c_int32 * MOEQ_PLAN_MAX_LEVELS),
                ("low_prime", ctypes.c_int32), ("low", ctypes.c_int32), ("floor", ctypes.c_int32),
                ("small_level", ctypes.c_int32), ("medium_level", ctypes.c_int32),
                ("small_params", ctypes.c_int64), ("medium_params", ctypes.c_int64),
                ("m_limit_bytes", ctypes.c_uint64), ("n_moe_layers", ctypes.c_int32)]


class moeq_plan_report(ctypes.Structure):
    _fields_ = [("s_low_gb", ctypes.c_double), ("b_base_gb", ctypes.c_double),
                ("b_delta_gb", ctypes.c_double), ("b_total_gb", ctypes.c_double),
                ("upgrade_gb", ctypes.c_double), ("total_gb", ctypes.c_double),
                ("n_upgraded", ctypes.c_int32), ("n_rule2", ctypes.c_int32),
                ("n_rule3", ctypes.c_int32), ("feasible", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    # torch ships its own HIP runtime under the same soname; loading torch first
    # makes libmoeq.so bind to that one instead of starting a second runtime
    # in the process (which then sees no device).
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    sig = {
        "moeq_layer_create": [ctypes.POINTER(moeq_config), P, P, P, P, I32, ctypes.POINTER(P)],
        "moeq_forward": [P, P, P, I32, P, P],
        "moeq_destroy": [P],
        "moeq_last_error": [],
        "moeq_set_path": [P, I32],
        "moeq_route": [P, P, I32, P, P, P],
        "moeq_bucket": [P, P, I32, P, P, P],
        "moeq_dequant": [P, I32, I32, P, P],
        "moeq_dequant_as": [P, I32, I32, I32, P, P],
        "moeq_quantize": [P, I32, I32, I32, P, P, P],
        "moeq_layer_bytes": [P, ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint64)],
        "moeq_set_stage_events": [P, ctypes.POINTER(P), I32],
        "moeq_set_router_weight": [P, P, I32],
        "moeq_sensitivity": [I32, ctypes.c_double, P, P, P, P],
        "moeq_layer_order": [I32, P],
        "moeq_plan_bits": [ctypes.POINTER(moeq_plan_params), I32, P, P, P, P, P,
                           ctypes.POINTER(moeq_plan_report)],
        "moeq_router_logits": [P, P, I32, P, P],
        "moeq_expert_importance": [ctypes.POINTER(moeq_config), P, P, I32, ctypes.c_double, ctypes.c_double,
                                   P, P, P, P],
        "moeq_expert_importance_noalloc": [ctypes.POINTER(moeq_config), P, P, I32, ctypes.c_double,
                                           ctypes.c_double, P, P, P, P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int32
    lib.moeq_destroy.restype = None
    lib.moeq_last_error.restype = ctypes.c_char_p
    return lib


lib = _load()


def header_functions():
    """Names of every function the public header declares."""
    with open(HEADER_PATH) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:moeq_status|void|const char\*)\s+(moeq_\w+)\s*\(",
                                 text, re.M)))


def moeq_last_error():
    return lib.moeq_last_error().decode()


def _check(status):
    if status != MOEQ_OK:
        raise MoeqError(status, moeq_last_error())


def moeq_layer_create(cfg, expert_mask, score_bias, routed, shared, weights_location):
    """cfg: moeq_config; expert_mask/score_bias: host addresses (score_bias may be 0);
    routed/shared: ctypes arrays of moeq_qtensor (shared may be None).  Returns the handle."""
    out = ctypes.c_void_p()
    _check(lib.moeq_layer_create(ctypes.byref(cfg), expert_mask, score_bias or None,
                                 routed, shared, weights_location, ctypes.byref(out)))
    return out.value


def moeq_forward(layer, x, logits, n_tokens, y, stream=0):
    _check(lib.moeq_forward(layer, x, logits, n_tokens, y, stream or None))


def moeq_set_router_weight(layer, w, location):
    _check(lib.moeq_set_router_weight(layer, w or None, location))


def moeq_router_logits(layer, x, n_tokens, logits, stream=0):
    _check(lib.moeq_router_logits(layer, x, n_tokens, logits, stream or None))


def moeq_sensitivity(ppl_low, ppl_high, params, layer_params):
    """-> numpy float64 [n]: Sens(t) for every tensor."""
    import numpy as np
    ph = np.ascontiguousarray(ppl_high, dtype=np.float64)
    pa = np.ascontiguousarray(params, dtype=np.int64)
    lp = np.ascontiguousarray(layer_params, dtype=np.int64)
    out = np.empty(len(ph), np.float64)
    _check(lib.moeq_sensitivity(len(ph), float(ppl_low), ph.ctypes.data, pa.ctypes.data, lp.ctypes.data,
                                out.ctypes.data))
    return out


def moeq_layer_order(n_layers):
    import numpy as np
    out = np.empty(max(n_layers, 0), np.int32)
    _check(lib.moeq_layer_order(n_layers, out.ctypes.data if n_layers > 0 else None))
    return out


def plan_params(*, ladder, low_prime, low, floor, small_level, medium_level, m_limit_bytes, n_moe_layers,
                small_params=10_000_000, medium_params=50_000_000):
    p = moeq_plan_params()
    p.n_levels = len(ladder)
    for i, v in enumerate(ladder[:MOEQ_PLAN_MAX_LEVELS]):
        p.width64[i] = int(v)
    p.low_prime, p.low, p.floor = low_prime, low, floor
    p.small_level, p.medium_level = small_level, medium_level
    p.small_params, p.medium_params = small_params, medium_params
    p.m_limit_bytes, p.n_moe_layers = m_limit_bytes, n_moe_layers
    return p


def moeq_plan_bits(p, params, sens, kind, layer):
    """-> (levels numpy int32 [n], moeq_plan_report)."""
    import numpy as np
    pa = np.ascontiguousarray(params, dtype=np.int64)
    se = np.ascontiguousarray(sens, dtype=np.float64)
    ki = np.ascontiguousarray(kind, dtype=np.int32)
    la = None if layer is None else np.ascontiguousarray(layer, dtype=np.int32)
    levels = np.empty(len(pa), np.int32)
    rep = moeq_plan_report()
    _check(lib.moeq_plan_bits(ctypes.byref(p), len(pa), pa.ctypes.data, se.ctypes.data, ki.ctypes.data,
                              None if la is None else la.ctypes.data, levels.ctypes.data, ctypes.byref(rep)))
    return levels, rep


def moeq_destroy(layer):
    lib.moeq_destroy(layer)


def moeq_set_path(layer, path):
    _check(lib.moeq_set_path(layer, path))


def moeq_route(layer, logits, n_tokens, idx, w, stream=0):
    _check(lib.moeq_route(layer, logits, n_tokens, idx, w, stream or None))


def moeq_bucket(layer, idx, n_tokens, offsets, perm, stream=0):
    _check(lib.moeq_bucket(layer, idx, n_tokens, offsets, perm, stream or None))


def moeq_dequant(layer, expert, proj, out, stream=0):
    _check(lib.moeq_dequant(layer, expert, proj, out, stream or None))


def moeq_dequant_as(layer, expert, proj, decoder, out, stream=0):
    _check(lib.moeq_dequant_as(layer, expert, proj, decoder, out, stream or None))


def moeq_quantize(w, rows, K, bits, codes, scales, stream=0):
    _check(lib.moeq_quantize(w, rows, K, bits, codes, scales, stream or None))


MOEQ_STAGE_EVENTS = 5


def moeq_set_stage_events(layer, events):
    """events: sequence of MOEQ_STAGE_EVENTS hipEvent_t handles (ints), or None to stop."""
    if not events:
        _check(lib.moeq_set_stage_events(layer, None, 0))
        return
    arr = (ctypes.c_void_p * len(events))(*events)
    _check(lib.moeq_set_stage_events(layer, arr, len(events)))


def moeq_expert_importance(cfg, score_bias, logits, n_tokens, alpha, retain, importance, mask, counts=0,
                           stream=0):
    """cfg: moeq_config; score_bias: host address or 0; the rest device addresses (counts may be 0)."""
    _check(lib.moeq_expert_importance(ctypes.byref(cfg), score_bias or None, logits, n_tokens, alpha, retain,
                                      importance, mask, counts or None, stream or None))


def moeq_expert_importance_noalloc(cfg, score_bias, logits, n_tokens, alpha, retain, importance, mask, counts=0,
                                   stream=0):
    """As moeq_expert_importance, with the library's static scratch (no allocation)."""
    _check(lib.moeq_expert_importance_noalloc(ctypes.byref(cfg), score_bias or None, logits, n_tokens, alpha,
                                              retain, importance, mask, counts or None, stream or None))


def expert_importance(shape, logits, *, alpha, retain, bias=None, stream=None):
    """Router-statistics importance and pruning mask (Section 3.1) for calibration
    logits (float32 CUDA tensor [n, E]) -> (importance float64, mask uint8, counts int32)."""
    import numpy as np
    import torch
    n, E = logits.shape
    cfg = make_config(shape, max_tokens=1)
    imp = torch.empty(E, dtype=torch.float64, device=logits.device)
    mask = torch.empty(E, dtype=torch.uint8, device=logits.device)
    counts = torch.empty(E, dtype=torch.int32, device=logits.device)
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    moeq_expert_importance(cfg, 0 if b is None else b.ctypes.data, logits.data_ptr(), n, float(alpha), float(retain),
                           imp.data_ptr(), mask.data_ptr(), counts.data_ptr(),
                           stream if stream is not None else torch.cuda.current_stream().cuda_stream)
    return imp, mask, counts


def moeq_layer_bytes(layer):
    wb, wsb = ctypes.c_uint64(), ctypes.c_uint64()
    _check(lib.moeq_layer_bytes(layer, ctypes.byref(wb), ctypes.byref(wsb)))
    return wb.value, wsb.value


# ---------------------------------------------------------------------------
def make_config(shape, max_tokens, decode_max_tokens=0):
    """A moeq_config from any object with the layer-shape attribute names."""
    return moeq_config(shape.hidden, shape.inter, shape.n_experts, shape.n_shared, shape.n_group,
                       shape.topk_group, shape.top_k, shape.group_topn, shape.norm_topk,
                       shape.routed_scale, max_tokens, decode_max_tokens, int(getattr(shape, "regroup", 0)))


def _addr(a):
    """Address of a numpy array or torch tensor (0 for None)."""
    if a is None:
        return 0
    if hasattr(a, "data_ptr"):
        return a.data_ptr()
    return a.ctypes.data


class Layer:
    """Owns one moeq layer handle.

    routed: dict expert -> (gate, up, down), each a dict with ``bits``,
    ``codes`` and ``scales`` (numpy arrays for host weights, torch device
    tensors for device weights); shared: list of such triples."""

    def __init__(self, shape, mask, routed, shared, *, max_tokens, bias=None,
                 decode_max_tokens=0, device_weights=False):
        import numpy as np
        self.shape = shape
        self.cfg = make_config(shape, max_tokens, decode_max_tokens)
        self._mask = np.ascontiguousarray(mask, dtype=np.uint8)
        self._bias = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        E, S = shape.n_experts, shape.n_shared
        r = (moeq_qtensor * (3 * E))()
        for e, triple in routed.items():
            for p, t in enumerate(triple):
                r[3 * e + p] = moeq_qtensor(int(t["bits"]), _addr(t["codes"]), _addr(t["scales"]))
        s = (moeq_qtensor * max(1, 3 * S))()
        for i, triple in enumerate(shared):
            for p, t in enumerate(triple):
                s[3 * i + p] = moeq_qtensor(int(t["bits"]), _addr(t["codes"]), _addr(t["scales"]))
        loc = MOEQ_WEIGHTS_DEVICE if device_weights else MOEQ_WEIGHTS_HOST
        self.device = None
        try:
            import torch
            if torch.cuda.is_available():
                self.device = torch.cuda.current_device()
        except ImportError:
            pass
        self.handle = moeq_layer_create(self.cfg, self._mask.ctypes.data,
                                        0 if self._bias is None else self._bias.ctypes.data,
                                        r, s if S else None, loc)

    def close(self):
        if getattr(self, "handle", None):
            moeq_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check_tensor(self, name, t, dtype, shape):
        """Shape, dtype, layout and device of a tensor handed to the library:
        the kernels trust these, and a wrong one would make them read or
        write outside the buffer."""
        import torch
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch tensor")
        if t.dtype != dtype:
            raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if t.device.type != "cuda" or (self.device is not None and t.device.index != self.device):
            raise ValueError(f"{name} must be on cuda:{self.device}, got {t.device}")

    @staticmethod
    def _stream(stream):
        if stream is not None:
            return stream
        import torch
        return torch.cuda.current_stream().cuda_stream

    def forward(self, x, logits=None, y=None, stream=None):
        """x: bf16 CUDA tensor [n, H]; logits: float32 CUDA tensor [n, E], or None
        to let the layer compute them with its router weight -> y float32 [n, H]."""
        import torch
        n = x.shape[0] if x.dim() == 2 else -1
        self._check_tensor("x", x, torch.bfloat16, (n, self.shape.hidden))
        if logits is not None:
            self._check_tensor("logits", logits, torch.float32, (n, self.shape.n_experts))
        if y is None:
            y = torch.empty((n, self.shape.hidden), dtype=torch.float32, device=x.device)
        self._check_tensor("y", y, torch.float32, (n, self.shape.hidden))
        moeq_forward(self.handle, x.data_ptr(), 0 if logits is None else logits.data_ptr(), n,
                     y.data_ptr(), self._stream(stream))
        return y

    def set_router_weight(self, w):
        """w: float32 [E, H], a numpy array (host) or CUDA tensor (device); None removes it."""
        if w is None:
            moeq_set_router_weight(self.handle, 0, MOEQ_WEIGHTS_HOST)
            return
        if hasattr(w, "data_ptr"):
            self._router_w = w.contiguous()
            moeq_set_router_weight(self.handle, self._router_w.data_ptr(), MOEQ_WEIGHTS_DEVICE)
        else:
            import numpy as np
            self._router_w = np.ascontiguousarray(w, dtype=np.float32)
            moeq_set_router_weight(self.handle, self._router_w.ctypes.data, MOEQ_WEIGHTS_HOST)
        self._router_w = None

    def router_logits(self, x, stream=None):
        """x: bf16 CUDA tensor [n, H] -> float32 logits [n, E] from the set router weight."""
        import torch
        n = x.shape[0] if x.dim() == 2 else -1
        self._check_tensor("x", x, torch.bfloat16, (n, self.shape.hidden))
        out = torch.empty((n, self.shape.n_experts), dtype=torch.float32, device=x.device)
        moeq_router_logits(self.handle, x.data_ptr(), n, out.data_ptr(), self._stream(stream))
        return out

    def route(self, logits, stream=None):
        import torch
        n = logits.shape[0] if logits.dim() == 2 else -1
        self._check_tensor("logits", logits, torch.float32, (n, self.shape.n_experts))
        idx = torch.empty((n, self.shape.top_k), dtype=torch.int32, device=logits.device)
        w = torch.empty((n, self.shape.top_k), dtype=torch.float32, device=logits.device)
        moeq_route(self.handle, logits.data_ptr(), n, idx.data_ptr(), w.data_ptr(),
                   self._stream(stream))
        return idx, w

    def bucket(self, idx, stream=None):
        import torch
        n = idx.shape[0] if idx.dim() == 2 else -1
        self._check_tensor("idx", idx, torch.int32, (n, self.shape.top_k))
        offsets = torch.empty(self.shape.n_experts + 1, dtype=torch.int32, device=idx.device)
        perm = torch.empty(n * self.shape.top_k, dtype=torch.int32, device=idx.device)
        moeq_bucket(self.handle, idx.data_ptr(), n, offsets.data_ptr(), perm.data_ptr(),
                    self._stream(stream))
        return offsets, perm

    def dequant(self, expert, proj, stream=None):
        import torch
        rows, K = self.shape.rows_cols(proj)
        out = torch.empty((rows, K), dtype=torch.float32, device="cuda")
        moeq_dequant(self.handle, expert, proj, out.data_ptr(), self._stream(stream))
        return out

    def dequant_as(self, expert, proj, decoder, stream=None):
        """One tensor through one of the library's decoders: float32 [rows, K]
        (MOEQ_DECODER_EXACT, MOEQ_DECODER_GEMV_SUBNORMAL) or binary16 bit
        patterns as int16 [rows, K] (MOEQ_DECODER_GEMM_F16)."""
        import torch
        rows, K = self.shape.rows_cols(proj)
        dt = torch.int16 if decoder == MOEQ_DECODER_GEMM_F16 else torch.float32
        out = torch.empty((rows, K), dtype=dt, device="cuda")
        moeq_dequant_as(self.handle, expert, proj, decoder, out.data_ptr(), self._stream(stream))
        return out

    def set_path(self, path):
        moeq_set_path(self.handle, path)

    def bytes(self):
        return moeq_layer_bytes(self.handle)


def quantize(w, bits, stream=None):
    """float32 CUDA tensor [rows, K] -> (codes uint8 [rows, K*bits/8], scales int16 [rows, K/32])."""
    import torch
    rows, K = w.shape
    codes = torch.empty((rows, K * bits // 8), dtype=torch.uint8, device=w.device)
    scales = torch.empty((rows, K // 32), dtype=torch.int16, device=w.device)
    moeq_quantize(w.data_ptr(), rows, K, bits, codes.data_ptr(), scales.data_ptr(),
                  stream if stream is not None else torch.cuda.current_stream().cuda_stream)
    return codes, scales
