"""ctypes binding of libspecverify.so.

Argument marshalling only: tensors are turned into device pointers and
element strides, the current HIP stream is passed through, and every step of
the computation runs in the library's kernels.  PyTorch provides device
memory and streams.  There is no fallback: if the library is missing or a
call fails, an exception is raised.
"""

import ctypes
import os
import threading

import torch  # loaded first so the library binds to the HIP runtime torch already loaded

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libspecverify.so"

SPEC_F32 = 0
SPEC_BF16 = 1
SPEC_TV_E2E = 0
SPEC_TV_PROD = 1
SPEC_TV_PER_STEP = 2
MODES = {"e2e": SPEC_TV_E2E, "prod": SPEC_TV_PROD, "per_step": SPEC_TV_PER_STEP}
STATUS = {0: "SPEC_OK", 1: "SPEC_EINVAL", 2: "SPEC_EUNSUPPORTED", 4: "SPEC_EWORKSPACE", 5: "SPEC_EHIP"}

_lib = None
_lock = threading.Lock()
_workspaces = {}

_c = ctypes
_P = _c.c_void_p
_I64 = _c.c_int64
_I = _c.c_int
_U64 = _c.c_uint64
_F = _c.c_float
_SZ = _c.c_size_t

VERIFY_ARGTYPES = [_P, _I64, _I64, _P, _I64, _I64, _I, _I, _I, _I, _P, _P, _F, _U64, _U64,
                   _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]
TV_ARGTYPES = [_P, _I64, _I64, _P, _I64, _I64, _I, _I, _I, _I, _F, _I, _F, _P, _P, _P, _P, _SZ, _P]
TO_ARGTYPES = [_P, _I64, _I64, _I, _I, _I, _I, _P, _P, _F, _U64, _U64, _P, _P, _P, _P, _P, _SZ, _P]
SAMPLE_ARGTYPES = [_P, _I64, _I, _I, _I, _P, _F, _U64, _U64, _P, _P, _P, _SZ, _P]
SAMPLE_GUMBEL_ARGTYPES = [_P, _I64, _I, _I, _I, _P, _F, _U64, _U64, _P, _P, _SZ, _P]
DIAG_ARGTYPES = [_P, _I64, _I64, _P, _I64, _I64, _I, _I, _I, _I, _P, _F, _P, _P, _P, _P, _SZ, _P]

# spec_launch: launch controls of spec_verify_ex
PATHS = {"auto": 0, "chain": 1, "single_read": 2}


class SpecLaunch(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int), ("groups", ctypes.c_int), ("residual_shape", ctypes.c_int)]


RESIDUAL_SHAPES = {"auto": 0, "wave": 1, "workgroup": 2}


VERIFY_EX_ARGTYPES = VERIFY_ARGTYPES + [ctypes.POINTER(SpecLaunch)]
# spec_verify_noalloc: spec_verify without the workspace pointer and size
VERIFY_NOALLOC_ARGTYPES = VERIFY_ARGTYPES[:-3] + [_P]
KL_ARGTYPES = [_P, _I64, _I64, _P, _I64, _I64, _I, _I, _I, _I, _F, _I, _F, _P, _P, _P, _P, _SZ, _P]
KL_KINDS = {"forward": 0, "ce": 1, "reverse": 2}
DIAG_COLUMNS = ("entropy_target", "entropy_draft", "max_p", "alpha_to", "alpha_rs", "alpha_p_gt_q", "alpha_q_ge_p")


class SpecError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__("%s failed: %s (%d)" % (fn, STATUS.get(status, "?"), status))
        self.status = status


def library_path():
    return os.environ.get("SPECVERIFY_LIB", os.path.join(HERE, _LIB_NAME))


def load_library():
    """Load libspecverify.so (once).  Raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError("%s not found: build it with `python -m paper_2606_12370_amd.build`" % path)
        lib = ctypes.CDLL(path)
        lib.spec_version.restype = _I
        lib.spec_status_string.restype = _c.c_char_p
        lib.spec_status_string.argtypes = [_I]
        lib.spec_verify_workspace_size.restype = _SZ
        lib.spec_verify_workspace_size.argtypes = [_I, _I, _I, _I]
        lib.spec_tv_workspace_size.restype = _SZ
        lib.spec_tv_workspace_size.argtypes = [_I, _I, _I, _I]
        lib.spec_verify.restype = _I
        lib.spec_verify.argtypes = VERIFY_ARGTYPES
        lib.spec_verify_ex.restype = _I
        lib.spec_verify_ex.argtypes = VERIFY_EX_ARGTYPES
        lib.spec_verify_noalloc.restype = _I
        lib.spec_verify_noalloc.argtypes = VERIFY_NOALLOC_ARGTYPES
        lib.spec_verify_noalloc_max_workspace.restype = _SZ
        lib.spec_verify_noalloc_max_workspace.argtypes = []
        lib.spec_tv_loss_fwd_bwd.restype = _I
        lib.spec_tv_loss_fwd_bwd.argtypes = TV_ARGTYPES
        lib.spec_verify_target_only_workspace_size.restype = _SZ
        lib.spec_verify_target_only_workspace_size.argtypes = [_I, _I, _I, _I]
        lib.spec_verify_target_only.restype = _I
        lib.spec_verify_target_only.argtypes = TO_ARGTYPES
        lib.spec_sample_workspace_size.restype = _SZ
        lib.spec_sample_workspace_size.argtypes = [_I, _I, _I]
        lib.spec_sample.restype = _I
        lib.spec_sample.argtypes = SAMPLE_ARGTYPES
        lib.spec_diagnostics_workspace_size.restype = _SZ
        lib.spec_diagnostics_workspace_size.argtypes = [_I, _I, _I, _I]
        lib.spec_diagnostics.restype = _I
        lib.spec_diagnostics.argtypes = DIAG_ARGTYPES
        lib.spec_verify_gumbel_workspace_size.restype = _SZ
        lib.spec_verify_gumbel_workspace_size.argtypes = [_I, _I, _I, _I]
        lib.spec_verify_gumbel.restype = _I
        lib.spec_verify_gumbel.argtypes = VERIFY_ARGTYPES
        lib.spec_sample_gumbel_workspace_size.restype = _SZ
        lib.spec_sample_gumbel_workspace_size.argtypes = [_I, _I, _I]
        lib.spec_sample_gumbel.restype = _I
        lib.spec_sample_gumbel.argtypes = SAMPLE_GUMBEL_ARGTYPES
        lib.spec_kl_workspace_size.restype = _SZ
        lib.spec_kl_workspace_size.argtypes = [_I, _I, _I, _I]
        lib.spec_kl_loss_fwd_bwd.restype = _I
        lib.spec_kl_loss_fwd_bwd.argtypes = KL_ARGTYPES
        _lib = lib
        return lib


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return SPEC_BF16
    if t.dtype == torch.float32:
        return SPEC_F32
    raise TypeError("logits must be bfloat16 or float32, got %s" % t.dtype)


def _ptr(t):
    return None if t is None else _P(t.data_ptr())


def _stream(device):
    return _P(torch.cuda.current_stream(device).cuda_stream)


def verify_gumbel_workspace_size(B, K, V, dtype=torch.bfloat16):
    code = SPEC_BF16 if dtype == torch.bfloat16 else SPEC_F32
    return int(load_library().spec_verify_gumbel_workspace_size(B, K, V, code))


def sample_gumbel_workspace_size(R, V, dtype=torch.bfloat16):
    code = SPEC_BF16 if dtype == torch.bfloat16 else SPEC_F32
    return int(load_library().spec_sample_gumbel_workspace_size(R, V, code))


def kl_workspace_size(N, K, V, dtype=torch.bfloat16):
    code = SPEC_BF16 if dtype == torch.bfloat16 else SPEC_F32
    return int(load_library().spec_kl_workspace_size(N, K, V, code))


def verify_workspace_size(B, K, V, dtype=torch.bfloat16):
    code = SPEC_BF16 if dtype == torch.bfloat16 else SPEC_F32
    return int(load_library().spec_verify_workspace_size(B, K, V, code))


def tv_workspace_size(N, K, V, dtype=torch.bfloat16):
    code = SPEC_BF16 if dtype == torch.bfloat16 else SPEC_F32
    return int(load_library().spec_tv_workspace_size(N, K, V, code))


def target_only_workspace_size(B, K, V, dtype=torch.bfloat16):
    code = SPEC_BF16 if dtype == torch.bfloat16 else SPEC_F32
    return int(load_library().spec_verify_target_only_workspace_size(B, K, V, code))


def sample_workspace_size(R, V, dtype=torch.bfloat16):
    code = SPEC_BF16 if dtype == torch.bfloat16 else SPEC_F32
    return int(load_library().spec_sample_workspace_size(R, V, code))


def diagnostics_workspace_size(B, K, V, dtype=torch.bfloat16):
    code = SPEC_BF16 if dtype == torch.bfloat16 else SPEC_F32
    return int(load_library().spec_diagnostics_workspace_size(B, K, V, code))


def _dev_key(device):
    device = torch.device(device)
    index = device.index if device.index is not None else torch.cuda.current_device()
    return (device.type, index)


def workspace(nbytes, device):
    """A scratch workspace of at least nbytes on `device`, cached per device
    and reused by every entry point and shape.  Calls that share it must be
    ordered on one stream (the current stream of each call)."""
    key = _dev_key(device)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
        _workspaces[key] = ws
    return ws


def _check_rows(t, name, shape):
    if t.dim() != 3 or tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if t.stride(2) != 1:
        raise ValueError("%s: the vocabulary dimension must be contiguous" % name)


def _temperature_arg(temperature, n):
    if torch.is_tensor(temperature):
        if temperature.dtype != torch.float32 or not temperature.is_contiguous() or temperature.numel() != n:
            raise ValueError("temperature tensor must be contiguous float32 [%d]" % n)
        return _ptr(temperature), 1.0
    return None, float(temperature)


def _check_ids(ids, B, K):
    if ids.dtype != torch.int32 or not ids.is_contiguous() or tuple(ids.shape) != (B, K):
        raise ValueError("draft_ids must be a contiguous int32 [B, K] tensor")


def verify(target_logits, draft_logits, draft_ids, temperature=1.0, seed=0, offset=0,
           want_debug=False, want_overlap=True, ws=None, out=None, gumbel=False, path=None, groups=0,
           noalloc=False, residual_shape=None):
    """Chain rejection-sampling verification (spec_verify, or with
    gumbel=True spec_verify_gumbel: the emitted token drawn by Gumbel-max).
    path ("auto", "chain", "single_read"), groups and residual_shape ("auto",
    "wave", "workgroup") select the launch (spec_verify_ex); by default the
    library chooses.  noalloc=True calls
    spec_verify_noalloc (the library's own scratch array, no workspace).

    target_logits [B, K+1, V], draft_logits [B, K, V] (bf16 or f32, same
    dtype, vocabulary dimension contiguous), draft_ids [B, K] int32,
    temperature: float or [B] float32 tensor.  Returns a dict with
    accept_len [B], emitted [B, K+1], overlap [B, K] (unless want_overlap is
    False, which lets the library skip most of the second read) and, with
    want_debug, p_at_draft, q_at_draft [B, K], logz_target [B, K+1],
    logz_draft [B, K].
    All work is enqueued on the current stream; nothing synchronises.
    """
    lib = load_library()
    B, K1, V = target_logits.shape
    K = K1 - 1
    _check_rows(target_logits, "target_logits", (B, K + 1, V))
    _check_rows(draft_logits, "draft_logits", (B, K, V))
    if draft_logits.dtype != target_logits.dtype:
        raise TypeError("target and draft logits must share a dtype")
    dev = target_logits.device
    ids = draft_ids
    if ids.dtype != torch.int32 or not ids.is_contiguous() or tuple(ids.shape) != (B, K):
        raise ValueError("draft_ids must be a contiguous int32 [B, K] tensor")
    if torch.is_tensor(temperature):
        if temperature.dtype != torch.float32 or not temperature.is_contiguous() or temperature.numel() != B:
            raise ValueError("temperature tensor must be contiguous float32 [B]")
        t_ptr, t_scalar = _ptr(temperature), 1.0
    else:
        t_ptr, t_scalar = None, float(temperature)
    code = _dtype_code(target_logits)
    if out is None:
        out = {
            "accept_len": torch.empty(B, dtype=torch.int32, device=dev),
            "emitted": torch.empty((B, K + 1), dtype=torch.int32, device=dev),
        }
        if want_overlap:
            out["overlap"] = torch.empty((B, K), dtype=torch.float32, device=dev)
        if want_debug:
            out["p_at_draft"] = torch.empty((B, K), dtype=torch.float32, device=dev)
            out["q_at_draft"] = torch.empty((B, K), dtype=torch.float32, device=dev)
            out["logz_target"] = torch.empty((B, K + 1), dtype=torch.float32, device=dev)
            out["logz_draft"] = torch.empty((B, K), dtype=torch.float32, device=dev)
    if noalloc:
        if gumbel or path is not None or groups or residual_shape is not None:
            raise ValueError("spec_verify_noalloc takes no launch controls")
        st = lib.spec_verify_noalloc(
            _ptr(target_logits), target_logits.stride(0), target_logits.stride(1),
            _ptr(draft_logits), draft_logits.stride(0), draft_logits.stride(1),
            code, B, K, V, _ptr(ids), t_ptr, t_scalar, int(seed) & (2**64 - 1), int(offset) & (2**64 - 1),
            _ptr(out["accept_len"]), _ptr(out["emitted"]), _ptr(out.get("overlap")),
            _ptr(out.get("p_at_draft")), _ptr(out.get("q_at_draft")),
            _ptr(out.get("logz_target")), _ptr(out.get("logz_draft")), _stream(dev))
        if st != 0:
            raise SpecError("spec_verify_noalloc", st)
        return out
    size_fn = lib.spec_verify_gumbel_workspace_size if gumbel else lib.spec_verify_workspace_size
    fn, name = (lib.spec_verify_gumbel, "spec_verify_gumbel") if gumbel else (lib.spec_verify, "spec_verify")
    extra = ()
    if path is not None or groups or residual_shape is not None:
        if gumbel:
            raise ValueError("launch controls apply to spec_verify only")
        fn, name = lib.spec_verify_ex, "spec_verify_ex"
        extra = (ctypes.byref(SpecLaunch(PATHS[path or "auto"], int(groups),
                                         RESIDUAL_SHAPES[residual_shape or "auto"])),)
    need = int(size_fn(B, K, V, code))
    if need == 0:
        raise ValueError("unsupported verify shape B=%d K=%d V=%d" % (B, K, V))
    if ws is None:
        ws = workspace(need, dev)
    st = fn(
        _ptr(target_logits), target_logits.stride(0), target_logits.stride(1),
        _ptr(draft_logits), draft_logits.stride(0), draft_logits.stride(1),
        code, B, K, V, _ptr(ids), t_ptr, t_scalar, int(seed) & (2**64 - 1), int(offset) & (2**64 - 1),
        _ptr(out["accept_len"]), _ptr(out["emitted"]), _ptr(out.get("overlap")),
        _ptr(out.get("p_at_draft")), _ptr(out.get("q_at_draft")),
        _ptr(out.get("logz_target")), _ptr(out.get("logz_draft")),
        _ptr(ws), ws.numel(), _stream(dev), *extra)
    if st != 0:
        raise SpecError(name, st)
    return out


def tv_loss_fwd_bwd(target_logits, draft_logits, temperature=1.0, mode="e2e", scale=1.0,
                    want_grad=True, want_overlap=True, ws=None, grad_out=None):
    """Fused TV loss forward + gradient (spec_tv_loss_fwd_bwd).

    target_logits, draft_logits [N, K, V] (bf16 or f32).  Returns
    (loss [1] float32, overlap [N, K] float32 or None, grad [N, K, V] float32
    or None).  All work is enqueued on the current stream.
    """
    lib = load_library()
    N, K, V = target_logits.shape
    _check_rows(target_logits, "target_logits", (N, K, V))
    _check_rows(draft_logits, "draft_logits", (N, K, V))
    if draft_logits.dtype != target_logits.dtype:
        raise TypeError("target and draft logits must share a dtype")
    dev = target_logits.device
    code = _dtype_code(target_logits)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    overlap = torch.empty((N, K), dtype=torch.float32, device=dev) if want_overlap else None
    grad = None
    if want_grad:
        grad = grad_out if grad_out is not None else torch.empty((N, K, V), dtype=torch.float32, device=dev)
        if not grad.is_contiguous() or tuple(grad.shape) != (N, K, V) or grad.dtype != torch.float32:
            raise ValueError("grad_out must be a contiguous float32 [N, K, V] tensor")
    need = int(lib.spec_tv_workspace_size(N, K, V, code))
    if need == 0:
        raise ValueError("unsupported TV shape N=%d K=%d V=%d" % (N, K, V))
    if ws is None:
        ws = workspace(need, dev)
    st = lib.spec_tv_loss_fwd_bwd(
        _ptr(target_logits), target_logits.stride(0), target_logits.stride(1),
        _ptr(draft_logits), draft_logits.stride(0), draft_logits.stride(1),
        code, N, K, V, float(temperature), MODES[mode] if isinstance(mode, str) else int(mode), float(scale),
        _ptr(loss), _ptr(overlap), _ptr(grad), _ptr(ws), ws.numel(), _stream(dev))
    if st != 0:
        raise SpecError("spec_tv_loss_fwd_bwd", st)
    return loss, overlap, grad


def verify_target_only(target_logits, draft_ids, temperature=1.0, seed=0, offset=0, want_debug=False,
                       ws=None, out=None):
    """Target-only verification of greedy draft tokens (spec_verify_target_only).

    target_logits [B, K+1, V] (bf16 or f32, vocabulary dimension contiguous),
    draft_ids [B, K] int32 (the draft's greedy tokens), temperature: float or
    [B] float32 tensor.  Returns a dict with accept_len [B], emitted [B, K+1]
    and, with want_debug, p_at_draft [B, K] and logz_target [B, K+1].
    """
    lib = load_library()
    B, K1, V = target_logits.shape
    K = K1 - 1
    _check_rows(target_logits, "target_logits", (B, K + 1, V))
    _check_ids(draft_ids, B, K)
    dev = target_logits.device
    t_ptr, t_scalar = _temperature_arg(temperature, B)
    code = _dtype_code(target_logits)
    if out is None:
        out = {
            "accept_len": torch.empty(B, dtype=torch.int32, device=dev),
            "emitted": torch.empty((B, K + 1), dtype=torch.int32, device=dev),
        }
        if want_debug:
            out["p_at_draft"] = torch.empty((B, K), dtype=torch.float32, device=dev)
            out["logz_target"] = torch.empty((B, K + 1), dtype=torch.float32, device=dev)
    need = int(lib.spec_verify_target_only_workspace_size(B, K, V, code))
    if need == 0:
        raise ValueError("unsupported target-only shape B=%d K=%d V=%d" % (B, K, V))
    if ws is None:
        ws = workspace(need, dev)
    st = lib.spec_verify_target_only(
        _ptr(target_logits), target_logits.stride(0), target_logits.stride(1), code, B, K, V,
        _ptr(draft_ids), t_ptr, t_scalar, int(seed) & (2**64 - 1), int(offset) & (2**64 - 1),
        _ptr(out["accept_len"]), _ptr(out["emitted"]), _ptr(out.get("p_at_draft")),
        _ptr(out.get("logz_target")), _ptr(ws), ws.numel(), _stream(dev))
    if st != 0:
        raise SpecError("spec_verify_target_only", st)
    return out


def sample(logits, temperature=1.0, seed=0, offset=0, want_logz=False, ws=None, out=None):
    """Draft-stage sampling (spec_sample) of one token per row.

    logits [R, V] (bf16 or f32, vocabulary dimension contiguous, any row
    stride); temperature: float or [R] float32 tensor, 0 meaning greedy.
    Returns a dict with tokens [R] int32 and, with want_logz, logz [R].
    """
    lib = load_library()
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be [R, V] with a contiguous vocabulary dimension")
    R, V = logits.shape
    dev = logits.device
    t_ptr, t_scalar = _temperature_arg(temperature, R)
    code = _dtype_code(logits)
    if out is None:
        out = {"tokens": torch.empty(R, dtype=torch.int32, device=dev)}
        if want_logz:
            out["logz"] = torch.empty(R, dtype=torch.float32, device=dev)
    need = int(lib.spec_sample_workspace_size(R, V, code))
    if need == 0:
        raise ValueError("unsupported sample shape R=%d V=%d" % (R, V))
    if ws is None:
        ws = workspace(need, dev)
    st = lib.spec_sample(
        _ptr(logits), logits.stride(0), code, R, V, t_ptr, t_scalar,
        int(seed) & (2**64 - 1), int(offset) & (2**64 - 1),
        _ptr(out["tokens"]), _ptr(out.get("logz")), _ptr(ws), ws.numel(), _stream(dev))
    if st != 0:
        raise SpecError("spec_sample", st)
    return out


def diagnostics(target_logits, draft_logits, temperature=1.0, ws=None):
    """Per-step acceptance diagnostics (spec_diagnostics).

    target_logits [B, >= K, V] (the first K rows of each batch row are used),
    draft_logits [B, K, V].  Returns a dict with one [B, K] float32 tensor per
    name in DIAG_COLUMNS (views of one [B, K, 7] tensor, also returned as
    "table"), greedy_draft [B, K] int32 and rs_preferred [B, K] int32.
    """
    lib = load_library()
    B, K, V = draft_logits.shape
    if target_logits.dim() != 3 or target_logits.shape[0] != B or target_logits.shape[1] < K \
            or target_logits.shape[2] != V or target_logits.stride(2) != 1:
        raise ValueError("target_logits must be [B, >=K, V] with a contiguous vocabulary dimension")
    _check_rows(draft_logits, "draft_logits", (B, K, V))
    if draft_logits.dtype != target_logits.dtype:
        raise TypeError("target and draft logits must share a dtype")
    dev = target_logits.device
    t_ptr, t_scalar = _temperature_arg(temperature, B)
    code = _dtype_code(target_logits)
    table = torch.empty((B, K, len(DIAG_COLUMNS)), dtype=torch.float32, device=dev)
    greedy = torch.empty((B, K), dtype=torch.int32, device=dev)
    prefer = torch.empty((B, K), dtype=torch.int32, device=dev)
    need = int(lib.spec_diagnostics_workspace_size(B, K, V, code))
    if need == 0:
        raise ValueError("unsupported diagnostics shape B=%d K=%d V=%d" % (B, K, V))
    if ws is None:
        ws = workspace(need, dev)
    st = lib.spec_diagnostics(
        _ptr(target_logits), target_logits.stride(0), target_logits.stride(1),
        _ptr(draft_logits), draft_logits.stride(0), draft_logits.stride(1),
        code, B, K, V, t_ptr, t_scalar, _ptr(table), _ptr(greedy), _ptr(prefer),
        _ptr(ws), ws.numel(), _stream(dev))
    if st != 0:
        raise SpecError("spec_diagnostics", st)
    out = {name: table[..., c] for c, name in enumerate(DIAG_COLUMNS)}
    out.update(table=table, greedy_draft=greedy, rs_preferred=prefer)
    return out


def sample_gumbel(logits, temperature=1.0, seed=0, offset=0, ws=None, out=None):
    """Gumbel-max draft sampling (spec_sample_gumbel) of one token per row.

    logits [R, V] (bf16 or f32, vocabulary dimension contiguous, any row
    stride); temperature: float or [R] float32 tensor, 0 meaning greedy.
    Returns a dict with tokens [R] int32.
    """
    lib = load_library()
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be [R, V] with a contiguous vocabulary dimension")
    R, V = logits.shape
    dev = logits.device
    t_ptr, t_scalar = _temperature_arg(temperature, R)
    code = _dtype_code(logits)
    if out is None:
        out = {"tokens": torch.empty(R, dtype=torch.int32, device=dev)}
    need = int(lib.spec_sample_gumbel_workspace_size(R, V, code))
    if need == 0:
        raise ValueError("unsupported sample shape R=%d V=%d" % (R, V))
    if ws is None:
        ws = workspace(need, dev)
    st = lib.spec_sample_gumbel(
        _ptr(logits), logits.stride(0), code, R, V, t_ptr, t_scalar,
        int(seed) & (2**64 - 1), int(offset) & (2**64 - 1), _ptr(out["tokens"]), _ptr(ws), ws.numel(), _stream(dev))
    if st != 0:
        raise SpecError("spec_sample_gumbel", st)
    return out


def kl_loss_fwd_bwd(target_logits, draft_logits, temperature=1.0, kind="forward", scale=1.0, want_grad=True,
                    want_per_step=True, ws=None, grad_out=None):
    """CE / forward-KL / reverse-KL loss and gradient (spec_kl_loss_fwd_bwd).

    target_logits, draft_logits [N, K, V] (bf16 or f32); kind in KL_KINDS.
    Returns (loss [1], per_step [N, K] or None, grad [N, K, V] or None).
    """
    lib = load_library()
    N, K, V = target_logits.shape
    _check_rows(target_logits, "target_logits", (N, K, V))
    _check_rows(draft_logits, "draft_logits", (N, K, V))
    if draft_logits.dtype != target_logits.dtype:
        raise TypeError("target and draft logits must share a dtype")
    dev = target_logits.device
    code = _dtype_code(target_logits)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    per_step = torch.empty((N, K), dtype=torch.float32, device=dev) if want_per_step else None
    grad = None
    if want_grad:
        grad = grad_out if grad_out is not None else torch.empty((N, K, V), dtype=torch.float32, device=dev)
        if not grad.is_contiguous() or tuple(grad.shape) != (N, K, V) or grad.dtype != torch.float32:
            raise ValueError("grad_out must be a contiguous float32 [N, K, V] tensor")
    need = int(lib.spec_kl_workspace_size(N, K, V, code))
    if need == 0:
        raise ValueError("unsupported KL shape N=%d K=%d V=%d" % (N, K, V))
    if ws is None:
        ws = workspace(need, dev)
    st = lib.spec_kl_loss_fwd_bwd(
        _ptr(target_logits), target_logits.stride(0), target_logits.stride(1),
        _ptr(draft_logits), draft_logits.stride(0), draft_logits.stride(1),
        code, N, K, V, float(temperature), KL_KINDS[kind] if isinstance(kind, str) else int(kind), float(scale),
        _ptr(loss), _ptr(per_step), _ptr(grad), _ptr(ws), ws.numel(), _stream(dev))
    if st != 0:
        raise SpecError("spec_kl_loss_fwd_bwd", st)
    return loss, per_step, grad
