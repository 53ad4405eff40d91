"""Python binding of liblam (include/lam.h) -- argument marshalling only.

Every step of the hot path runs in the HIP library; this module only turns
torch tensors into device pointers and sizes, calls the C ABI through ctypes,
and turns status codes into exceptions.  torch provides device memory and the
current stream; nothing here computes on the CPU.  If the library has not been
built (``python paper_2609_32256_amd/build.py``) importing this module fails.

    import torch, paper_2609_32256_amd as lam
    codes, p = lam.quantize(x, eps=1e-3)            # Q_eps, packed b-bit codes
    xh = lam.dequantize(codes, p)
    s = lam.Store(dim=768, tau=0.95, capacity=1 << 20)
    rep, stats = s.ingest(x_batch)                 # greedy near-duplicate test
    s.quantize(eps=1e-3)
    scores, ids, bound = s.score_topk(q, k=10)
    s.score_topk_certified(q, k=10)                # + rank-invariance flags
    s.block_encode(); s.score_topk_blocks(q, 10)   # per-block codec of the codes
    lam.removal_ceiling(x, tau=0.95)               # greedy at delta and at 2 delta
    b = lam.Store(768, 0.95, 1 << 20, eps_band=0.2 / 768 ** 0.5, band_width=4)
                                                   # banded candidates over Q_eps codes
"""
from __future__ import annotations

import ctypes
import os
import torch  # noqa: F401  (loads the HIP runtime that liblam then shares)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblam.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2609_32256_amd/build.py`")

_lib = ctypes.CDLL(LIB_PATH)

STATUS = {0: "LAM_OK", 1: "LAM_EINVAL", 2: "LAM_ERANGE", 3: "LAM_ENOMEM", 4: "LAM_ECAPACITY",
          5: "LAM_EDEVICE", 6: "LAM_ESTATE"}
PACK_BITS, PACK_BYTES = 0, 1
_MODES = {"bits": PACK_BITS, "bytes": PACK_BYTES}


class LamError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status
        self.name = STATUS.get(status, str(status))


class QParams(ctypes.Structure):
    _fields_ = [("eps", ctypes.c_double), ("step", ctypes.c_double), ("absmax", ctypes.c_float),
                ("bits", ctypes.c_int32), ("mode", ctypes.c_int32), ("max_code", ctypes.c_int32),
                ("n", ctypes.c_int64), ("code_bytes", ctypes.c_uint64)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class IngestStats(ctypes.Structure):
    _fields_ = [("n_in", ctypes.c_int64), ("n_kept", ctypes.c_int64), ("n_dropped", ctypes.c_int64),
                ("store_size", ctypes.c_int64), ("n_ambiguous_pairs", ctypes.c_int64),
                ("n_exact_escalations", ctypes.c_int64), ("delta_hat_call", ctypes.c_double),
                ("delta_hat_run", ctypes.c_double), ("min_margin_d2", ctypes.c_double)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class StoreInfo(ctypes.Structure):
    _fields_ = [("size", ctypes.c_int64), ("capacity", ctypes.c_int64), ("n_seen", ctypes.c_int64),
                ("dim", ctypes.c_int32), ("quantized", ctypes.c_int32), ("tau", ctypes.c_double),
                ("delta_hat_run", ctypes.c_double), ("q", QParams)]


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
class BlockStats(ctypes.Structure):
    _fields_ = [("rows", _I64), ("blocks", _I64), ("data_bytes", ctypes.c_uint64), ("meta_bytes", ctypes.c_uint64),
                ("total_bytes", ctypes.c_uint64), ("bits_per_code", ctypes.c_double), ("plain_bits", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("codec_ratio", ctypes.c_double), ("composite_ratio", ctypes.c_double)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_ if f != "pad"}


class CeilingStats(ctypes.Structure):
    _fields_ = [("n", _I64), ("kept", _I64), ("kept_2delta", _I64), ("tau", ctypes.c_double),
                ("tau_2delta", ctypes.c_double), ("removal", ctypes.c_double), ("ceiling", ctypes.c_double),
                ("frac_of_ceiling", ctypes.c_double), ("bits_lo", ctypes.c_double), ("bits_hi", ctypes.c_double),
                ("delta_hat", ctypes.c_double), ("delta_hat_2delta", ctypes.c_double)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


_SIGS = {
    "lam_abi_version": ([], ctypes.c_int),
    "lam_status_name": ([ctypes.c_int], ctypes.c_char_p),
    "lam_last_error": ([], ctypes.c_char_p),
    "lam_ctx_create": ([ctypes.c_int, _P, ctypes.POINTER(_P)], ctypes.c_int),
    "lam_ctx_destroy": ([_P], None),
    "lam_ctx_synchronize": ([_P], ctypes.c_int),
    "lam_ctx_profile": ([_P, ctypes.c_int], ctypes.c_int),
    "lam_ctx_profile_only": ([_P, ctypes.c_char_p], ctypes.c_int),
    "lam_ctx_set_screen_tile": ([_P, ctypes.c_int], ctypes.c_int),
    "lam_ctx_profile_reset": ([_P], ctypes.c_int),
    "lam_ctx_profile_read": ([_P, ctypes.c_char_p, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_I64)],
                             ctypes.c_int),
    "lam_qeps_plan": ([ctypes.c_double, ctypes.c_float, ctypes.c_int, _I64, ctypes.POINTER(QParams)], ctypes.c_int),
    "lam_quantize": ([_P, _P, _I64, ctypes.c_double, ctypes.c_float, ctypes.c_int, _P, ctypes.c_uint64,
                      ctypes.POINTER(QParams)], ctypes.c_int),
    "lam_quantize_async": ([_P, _P, _I64, ctypes.c_double, ctypes.c_float, ctypes.c_int, _P, ctypes.c_uint64, _P,
                            ctypes.POINTER(QParams)], ctypes.c_int),
    "lam_dequantize": ([_P, _P, ctypes.POINTER(QParams), _P], ctypes.c_int),
    "lam_store_create": ([_P, ctypes.c_int32, ctypes.c_double, _I64, ctypes.POINTER(_P)], ctypes.c_int),
    "lam_store_create_banded": ([_P, ctypes.c_int32, ctypes.c_double, _I64, ctypes.c_double, ctypes.c_int32,
                                 ctypes.POINTER(_P)], ctypes.c_int),
    "lam_store_destroy": ([_P], None),
    "lam_store_get_info": ([_P, ctypes.POINTER(StoreInfo)], ctypes.c_int),
    "lam_dedup_ingest": ([_P, _P, _P, _I64, _P, _P, ctypes.POINTER(IngestStats)], ctypes.c_int),
    "lam_store_quantize": ([_P, _P, ctypes.c_double, ctypes.c_float, ctypes.c_int, ctypes.POINTER(QParams)],
                           ctypes.c_int),
    "lam_store_clear": ([_P, _P], ctypes.c_int),
    "lam_store_dequantize": ([_P, _P, _P], ctypes.c_int),
    "lam_store_export": ([_P, _P, _P, _P, ctypes.c_uint64], ctypes.c_int),
    "lam_score_topk_certified": ([_P, _P, _P, _I64, ctypes.c_int32, _P, _P, _P, _P, _P], ctypes.c_int),
    "lam_store_block_encode": ([_P, _P, ctypes.POINTER(BlockStats)], ctypes.c_int),
    "lam_store_block_decode": ([_P, _P, _P], ctypes.c_int),
    "lam_store_block_export": ([_P, _P, _P, _P, _P, ctypes.c_uint64], ctypes.c_int),
    "lam_score_topk_blocks": ([_P, _P, _P, _I64, ctypes.c_int32, _P, _P, _P], ctypes.c_int),
    "lam_removal_ceiling": ([_P, _P, _I64, ctypes.c_int32, ctypes.c_double, _I64, ctypes.POINTER(CeilingStats)],
                            ctypes.c_int),
    "lam_score_topk": ([_P, _P, _P, _I64, ctypes.c_int32, _P, _P, _P], ctypes.c_int),
    "lam_score_topk_noalloc": ([_P, _P, _P, _I64, ctypes.c_int32, _P, _P, _P], ctypes.c_int),
    "lam_triad": ([_P, _P, _P, _P, _I64, ctypes.c_float], ctypes.c_int),
}
for _name, (_args, _res) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = _res

EXPORTED = tuple(_SIGS)


def _check(status: int):
    if status != 0:
        raise LamError(status, _lib.lam_last_error().decode(errors="replace"))


def abi_version() -> int:
    return _lib.lam_abi_version()


def removal_ceiling(x: torch.Tensor, tau: float, batch: int = 4096, ctx: Context | None = None) -> dict:
    """Theorem "removal ceiling" / Corollary "measured bracket": greedy over the
    rows of x at tau and at 4 tau - 3 (radius 2 delta).  Returns the counts,
    the attained removal, the ceiling and the bracket log2|R(2 delta)| <=
    H_delta <= log2|R(delta)|."""
    ctx = ctx or default_context()
    x = _dev_tensor(x, torch.float32, "x")
    if x.dim() != 2:
        raise ValueError("x must be (n, dim)")
    out = CeilingStats()
    _check(_lib.lam_removal_ceiling(ctx.handle, _ptr(x), x.shape[0], x.shape[1], float(tau), int(batch),
                                    ctypes.byref(out)))
    return out.as_dict()


def qeps_plan(eps: float, absmax: float, mode: str = "bits", n: int = 0) -> QParams:
    """Width plan of Q_eps (host only)."""
    p = QParams()
    _check(_lib.lam_qeps_plan(float(eps), float(absmax), _MODES[mode], int(n), ctypes.byref(p)))
    return p


# ---------------------------------------------------------------- contexts
class Context:
    """A liblam context bound to one device and one HIP stream."""

    def __init__(self, device: int | None = None, stream: "torch.cuda.Stream | None" = None):
        if not torch.cuda.is_available():
            raise RuntimeError("liblam needs a GPU (torch.cuda.is_available() is False)")
        self.device = torch.cuda.current_device() if device is None else int(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        h = _P()
        _check(_lib.lam_ctx_create(self.device, _P(self.stream.cuda_stream), ctypes.byref(h)))
        self._h = h

    @property
    def handle(self):
        return self._h

    def synchronize(self):
        _check(_lib.lam_ctx_synchronize(self._h))

    def profile(self, enable: bool = True):
        _check(_lib.lam_ctx_profile(self._h, 1 if enable else 0))

    def profile_only(self, kernel: str | None):
        """Time only the launches of the kernel names in a comma-separated list
        (None: every kernel)."""
        _check(_lib.lam_ctx_profile_only(self._h, (kernel or "").encode()))

    def profile_reset(self):
        _check(_lib.lam_ctx_profile_reset(self._h))

    def set_screen_tile(self, policy):
        """The screen's tile: "auto" (by launch size), "small" (128 x 128) or
        "large" (256 x 256 where D is 768 or 1,024).  Decisions are the same."""
        code = {"auto": 0, "small": 1, "large": 2}.get(policy, policy)
        _check(_lib.lam_ctx_set_screen_tile(self._h, int(code)))

    def profile_read(self, kernel: str):
        ms, n = ctypes.c_double(), _I64()
        _check(_lib.lam_ctx_profile_read(self._h, kernel.encode(), ctypes.byref(ms), ctypes.byref(n)))
        return ms.value, n.value

    def close(self):
        if getattr(self, "_h", None):
            _lib.lam_ctx_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


_default_ctx: dict = {}


def default_context() -> Context:
    dev = torch.cuda.current_device()
    key = (dev, torch.cuda.current_stream(dev).cuda_stream)
    c = _default_ctx.get(key)
    if c is None:
        c = _default_ctx[key] = Context(dev)
    return c


def _ptr(t: torch.Tensor | None):
    return _P(t.data_ptr()) if t is not None else _P(None)


def _dev_tensor(t: torch.Tensor, dtype, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")
    return t.contiguous()


# ---------------------------------------------------------------- Q_eps
def quantize(x: torch.Tensor, eps: float, absmax: float | None = None, mode: str = "bits",
             out: torch.Tensor | None = None, ctx: Context | None = None):
    """Q_eps of a float32 tensor: returns (codes uint32-words tensor viewed as
    int32, QParams).  absmax=None measures max|x| on the device."""
    ctx = ctx or default_context()
    x = _dev_tensor(x, torch.float32, "x").reshape(-1)
    n = x.numel()
    a = 0.0 if absmax is None else float(absmax)
    if out is None:
        plan_a = a if absmax is not None else 0.0
        # capacity for the widest code the plan could pick (32 bits) if absmax is measured
        words = (n * 32 + 31) // 32 if absmax is None else (n * qeps_plan(eps, plan_a, mode, n).bits + 31) // 32
        out = torch.empty(max(1, words), dtype=torch.int32, device=x.device)
    p = QParams()
    _check(_lib.lam_quantize(ctx.handle, _ptr(x), n, float(eps), a, _MODES[mode], _ptr(out),
                             out.numel() * 4, ctypes.byref(p)))
    return out[: p.code_bytes // 4], p


def quantize_async(x: torch.Tensor, eps: float, absmax: float, status: torch.Tensor, mode: str = "bits",
                   out: torch.Tensor | None = None, ctx: Context | None = None):
    """Q_eps that does not wait for the device (lam_quantize_async): returns
    (codes, QParams) once the encode is queued; the encode adds a positive
    count to status[0] if any element is NaN/Inf and to status[1] if any is
    above absmax (status: a contiguous int32 device tensor of at least 2
    entries that the caller clears)."""
    ctx = ctx or default_context()
    x = _dev_tensor(x, torch.float32, "x").reshape(-1)
    if not isinstance(status, torch.Tensor) or not status.is_cuda or status.dtype != torch.int32 \
            or not status.is_contiguous() or status.numel() < 2:
        raise ValueError("status must be a contiguous int32 device tensor of at least 2 entries")
    n = x.numel()
    if out is None:
        out = torch.empty(max(1, (n * qeps_plan(eps, absmax, mode, n).bits + 31) // 32), dtype=torch.int32,
                          device=x.device)
    p = QParams()
    _check(_lib.lam_quantize_async(ctx.handle, _ptr(x), n, float(eps), float(absmax), _MODES[mode], _ptr(out),
                                   out.numel() * 4, _ptr(status), ctypes.byref(p)))
    return out[: p.code_bytes // 4], p


def dequantize(codes: torch.Tensor, p: QParams, out: torch.Tensor | None = None,
               ctx: Context | None = None) -> torch.Tensor:
    ctx = ctx or default_context()
    codes = _dev_tensor(codes, torch.int32, "codes")
    if codes.numel() * 4 < p.code_bytes:
        raise ValueError("codes tensor shorter than params.code_bytes")
    if out is None:
        out = torch.empty(p.n, dtype=torch.float32, device=codes.device)
    _check(_lib.lam_dequantize(ctx.handle, _ptr(codes), ctypes.byref(p), _ptr(out)))
    return out


def triad(a: torch.Tensor, b: torch.Tensor, c: torch.Tensor, s: float = 3.0, ctx: Context | None = None):
    """The bandwidth anchor c = a + s * b over float32 device tensors of equal
    size (lam_triad; 12 bytes moved per element)."""
    ctx = ctx or default_context()
    a = _dev_tensor(a, torch.float32, "a")
    b = _dev_tensor(b, torch.float32, "b")
    c = _dev_tensor(c, torch.float32, "c")
    if not (a.numel() == b.numel() == c.numel()):
        raise ValueError("a, b and c must have the same size")
    _check(_lib.lam_triad(ctx.handle, _ptr(a), _ptr(b), _ptr(c), a.numel(), float(s)))
    return c


# ---------------------------------------------------------------- store
class Store:
    """The retained set of the greedy near-duplicate test, on one device."""

    def __init__(self, dim: int, tau: float, capacity: int, ctx: Context | None = None,
                 eps_band: float | None = None, band_width: int | None = None):
        """With eps_band and band_width the store takes its candidates from a
        band index over Q_eps codes (lam_store_create_banded); otherwise every
        retained row is screened."""
        self.ctx = ctx or default_context()
        h = _P()
        if (eps_band is None) != (band_width is None):
            raise ValueError("give both eps_band and band_width, or neither")
        if band_width is None:
            _check(_lib.lam_store_create(self.ctx.handle, int(dim), float(tau), int(capacity), ctypes.byref(h)))
        else:
            _check(_lib.lam_store_create_banded(self.ctx.handle, int(dim), float(tau), int(capacity),
                                                float(eps_band), int(band_width), ctypes.byref(h)))
        self._h = h
        self.banded = band_width is not None
        self.dim = int(dim)
        self.tau = float(tau)

    def info(self) -> StoreInfo:
        i = StoreInfo()
        _check(_lib.lam_store_get_info(self._h, ctypes.byref(i)))
        return i

    @property
    def size(self) -> int:
        return self.info().size

    def ingest(self, x: torch.Tensor, max_cos: bool = False, rep: torch.Tensor | None = None, sync: bool = True):
        """Algorithm "admit" over the rows of x (n x dim float32).  Returns
        (rep int64[n], stats dict[, max_cos float32[n]]).  With sync=False the
        call may return before the device has finished (stats is then None);
        invalid input of such a call is raised by the next call that waits
        (size, info, quantize, scoring or a synchronous ingest)."""
        x = _dev_tensor(x, torch.float32, "x")
        if x.dim() != 2 or x.shape[1] != self.dim:
            raise ValueError(f"x must be (n, {self.dim})")
        n = x.shape[0]
        if rep is None:
            rep = torch.empty(n, dtype=torch.int64, device=x.device)
        mc = torch.empty(n, dtype=torch.float32, device=x.device) if max_cos else None
        st = IngestStats() if sync else None
        _check(_lib.lam_dedup_ingest(self.ctx.handle, self._h, _ptr(x), n, _ptr(rep), _ptr(mc),
                                     ctypes.byref(st) if st is not None else None))
        stats = st.as_dict() if st is not None else None
        return (rep, stats, mc) if max_cos else (rep, stats)

    def quantize(self, eps: float, absmax: float | None = None, mode: str = "bits") -> QParams:
        p = QParams()
        _check(_lib.lam_store_quantize(self.ctx.handle, self._h, float(eps),
                                       0.0 if absmax is None else float(absmax), _MODES[mode], ctypes.byref(p)))
        return p

    def clear(self):
        """Empty the store, keeping its device memory."""
        _check(_lib.lam_store_clear(self.ctx.handle, self._h))

    def dequantize(self, out: torch.Tensor | None = None) -> torch.Tensor:
        """The reconstruction x_hat of every retained row (size x dim float32)."""
        n = self.size
        if out is None:
            out = torch.empty((max(1, n), self.dim), dtype=torch.float32, device=f"cuda:{self.ctx.device}")
        _check(_lib.lam_store_dequantize(self.ctx.handle, self._h, _ptr(out)))
        return out[:n]

    def ids(self) -> torch.Tensor:
        n = self.size
        out = torch.empty(max(1, n), dtype=torch.int64, device=f"cuda:{self.ctx.device}")
        _check(_lib.lam_store_export(self.ctx.handle, self._h, _ptr(out), _P(None), 0))
        return out[:n]

    def codes(self) -> torch.Tensor:
        p = self.info().q
        out = torch.empty(max(1, p.code_bytes // 4), dtype=torch.int32, device=f"cuda:{self.ctx.device}")
        _check(_lib.lam_store_export(self.ctx.handle, self._h, _P(None), _ptr(out), out.numel() * 4))
        return out[: p.code_bytes // 4]

    def block_encode(self) -> dict:
        """Per-block codec of the current codes (lam_store_block_encode)."""
        st = BlockStats()
        _check(_lib.lam_store_block_encode(self.ctx.handle, self._h, ctypes.byref(st)))
        self._blocks = st.as_dict()
        return self._blocks

    def block_decode(self, out: torch.Tensor | None = None) -> torch.Tensor:
        n = self.size
        if out is None:
            out = torch.empty((max(1, n), self.dim), dtype=torch.float32, device=f"cuda:{self.ctx.device}")
        _check(_lib.lam_store_block_decode(self.ctx.handle, self._h, _ptr(out)))
        return out[:n]

    def block_export(self):
        """(widths uint8[size, dim/32], row_off int64[size + 1], data int32[words])."""
        n = self.size
        dev = f"cuda:{self.ctx.device}"
        words = int(self._blocks["data_bytes"] // 4)
        w = torch.empty((max(1, n), self.dim // 32), dtype=torch.uint8, device=dev)
        ro = torch.empty(n + 1, dtype=torch.int64, device=dev)
        d = torch.empty(max(1, words), dtype=torch.int32, device=dev)
        _check(_lib.lam_store_block_export(self.ctx.handle, self._h, _ptr(w), _ptr(ro), _ptr(d), d.numel() * 4))
        return w[:n], ro, d[:words]

    def score_topk_blocks(self, q: torch.Tensor, k: int):
        """lam_score_topk over the block encoding."""
        q = _dev_tensor(q, torch.float32, "q")
        nq = q.shape[0]
        scores = torch.empty((nq, k), dtype=torch.float32, device=q.device)
        ids = torch.empty((nq, k), dtype=torch.int64, device=q.device)
        bound = torch.empty(nq, dtype=torch.float32, device=q.device)
        _check(_lib.lam_score_topk_blocks(self.ctx.handle, self._h, _ptr(q), nq, int(k), _ptr(scores), _ptr(ids),
                                          _ptr(bound)))
        return scores, ids, bound

    def score_topk_certified(self, q: torch.Tensor, k: int):
        """Top-k plus the rank-invariance certificate: (scores, ids, bound,
        certified bool[nq], margin float32[nq]); see lam_score_topk_certified."""
        q = _dev_tensor(q, torch.float32, "q")
        if q.dim() != 2 or q.shape[1] != self.dim:
            raise ValueError(f"q must be (nq, {self.dim})")
        nq = q.shape[0]
        dev = q.device
        scores = torch.empty((nq, k), dtype=torch.float32, device=dev)
        ids = torch.empty((nq, k), dtype=torch.int64, device=dev)
        bound = torch.empty(nq, dtype=torch.float32, device=dev)
        cert = torch.empty(nq, dtype=torch.uint8, device=dev)
        margin = torch.empty(nq, dtype=torch.float32, device=dev)
        _check(_lib.lam_score_topk_certified(self.ctx.handle, self._h, _ptr(q), nq, int(k), _ptr(scores), _ptr(ids),
                                             _ptr(bound), _ptr(cert), _ptr(margin)))
        return scores, ids, bound, cert.bool(), margin

    def score_topk(self, q: torch.Tensor, k: int, out=None):
        """Top-k (scores float32[nq, k], ids int64[nq, k], bound float32[nq])."""
        q = _dev_tensor(q, torch.float32, "q")
        if q.dim() != 2 or q.shape[1] != self.dim:
            raise ValueError(f"q must be (nq, {self.dim})")
        nq = q.shape[0]
        if out is None:
            out = (torch.empty((nq, k), dtype=torch.float32, device=q.device),
                   torch.empty((nq, k), dtype=torch.int64, device=q.device),
                   torch.empty(nq, dtype=torch.float32, device=q.device))
        s, i, b = out
        _check(_lib.lam_score_topk(self.ctx.handle, self._h, _ptr(q), nq, int(k), _ptr(s), _ptr(i), _ptr(b)))
        return s, i, b

    def score_topk_noalloc(self, q: torch.Tensor, k: int, out):
        """score_topk through the allocation-free entry point (lam_score_topk_noalloc):
        the library takes its scratch from a fixed per-device array; the caller
        passes every output, out = (scores float32[nq, k], ids int64[nq, k],
        bound float32[nq]).  nq <= 256; the store must be settled (info())."""
        q = _dev_tensor(q, torch.float32, "q")
        if q.dim() != 2 or q.shape[1] != self.dim:
            raise ValueError(f"q must be (nq, {self.dim})")
        s, i, b = out
        _check(_lib.lam_score_topk_noalloc(self.ctx.handle, self._h, _ptr(q), q.shape[0], int(k), _ptr(s), _ptr(i),
                                           _ptr(b)))
        return s, i, b

    def close(self):
        if getattr(self, "_h", None):
            _lib.lam_store_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


__all__ = ["LamError", "QParams", "IngestStats", "StoreInfo", "Context", "default_context", "quantize",
           "dequantize", "triad", "Store", "qeps_plan", "removal_ceiling", "CeilingStats", "abi_version", "EXPORTED", "LIB_PATH"]
