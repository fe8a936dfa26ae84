"""Stream-CQSA hot path for AMD MI355X: thin ctypes binding of libcqsa.so.

The binding only marshals arguments: every step of planning and compute runs
in the native library (C++ planner, HIP kernels for gfx950).  PyTorch is used
for device memory and streams.  The binding fails loudly when the library has
not been built (``python -m paper_2604_20819_amd.build``); there is no CPU or
eager fallback.

Names follow include/cqsa.h: ``cqsa_plan``, ``cqsa_forward``,
``cqsa_backward``, ``cqsa_set_timing``, ``cqsa_last_stats`` ...
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libcqsa.so")

CQSA_F32, CQSA_F16, CQSA_BF16 = 0, 1, 2
CQSA_MEM_HOST, CQSA_MEM_DEVICE = 0, 1
STATUS = {0: "CQSA_OK", -1: "CQSA_ERR_INVALID_ARG", -2: "CQSA_ERR_UNSUPPORTED",
          -3: "CQSA_ERR_BUDGET", -4: "CQSA_ERR_DEVICE_OOM", -5: "CQSA_ERR_HIP",
          -6: "CQSA_ERR_INTERNAL"}


class CqsaError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class cqsa_tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int), ("where", ctypes.c_int),
                ("B", ctypes.c_int64), ("L", ctypes.c_int64), ("H", ctypes.c_int64),
                ("d", ctypes.c_int64)]


class cqsa_interest_set(ctypes.Structure):
    _fields_ = [("c", ctypes.c_int32), ("l", ctypes.c_int32), ("interest", ctypes.c_int32 * 16)]


class cqsa_plan_opts(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("dtype", ctypes.c_int), ("c", ctypes.c_int32),
                ("l", ctypes.c_int32), ("interest", ctypes.c_int32 * 16),
                ("depth", ctypes.c_int32), ("min_depth", ctypes.c_int32),
                ("max_depth", ctypes.c_int32), ("n_slots", ctypes.c_int32),
                ("inputs_on_device", ctypes.c_int32), ("acc_on_device", ctypes.c_int32),
                ("with_backward", ctypes.c_int32), ("tasks_per_slot", ctypes.c_int32),
                ("n_level_sets", ctypes.c_int32), ("level_sets", cqsa_interest_set * 4),
                ("read_in_place", ctypes.c_int32),
                ("out16", ctypes.c_int32), ("bwd_tasks_per_launch", ctypes.c_int32)]


class cqsa_run(ctypes.Structure):
    _fields_ = [("global_start", ctypes.c_int64), ("length", ctypes.c_int64),
                ("bits", ctypes.c_uint32)]


class cqsa_task(ctypes.Structure):
    _fields_ = [("index", ctypes.c_int64), ("depth", ctypes.c_int32),
                ("quorum", ctypes.POINTER(ctypes.c_int32)), ("L_local", ctypes.c_int64),
                ("n_runs", ctypes.c_int32), ("runs", ctypes.POINTER(cqsa_run)),
                ("n_blocks", ctypes.c_int64), ("block_or", ctypes.POINTER(ctypes.c_uint32)),
                ("block_and", ctypes.POINTER(ctypes.c_uint32))]


class cqsa_run_stats(ctypes.Structure):
    _fields_ = [("depth", ctypes.c_int32), ("num_tasks", ctypes.c_int64),
                ("modelled_device_bytes", ctypes.c_uint64), ("workspace_bytes", ctypes.c_uint64),
                ("h2d_bytes", ctypes.c_uint64), ("d2h_bytes", ctypes.c_uint64),
                ("d2d_bytes", ctypes.c_uint64), ("inner_launches", ctypes.c_int64),
                ("ms_wall", ctypes.c_double), ("ms_stage", ctypes.c_double),
                ("ms_inner", ctypes.c_double), ("ms_merge", ctypes.c_double),
                ("ms_finalize", ctypes.c_double), ("ms_d2h", ctypes.c_double),
                ("tiles_full", ctypes.c_int64), ("tiles_clear", ctypes.c_int64),
                ("tiles_mixed", ctypes.c_int64), ("merge_launches", ctypes.c_int64),
                ("ms_inner_busy", ctypes.c_double), ("guard_steps", ctypes.c_int64),
                ("resident_tasks", ctypes.c_int64), ("kernel_tiles_masked", ctypes.c_int64),
                ("kernel_tiles_clear", ctypes.c_int64), ("kernel_tiles_mixed", ctypes.c_int64),
                ("kernel_kv_tiles_masked", ctypes.c_int64), ("kernel_kv_tiles_clear", ctypes.c_int64),
                ("kernel_kv_tiles_mixed", ctypes.c_int64)]


# Every symbol include/cqsa.h declares, with its ctypes signature.
_SIGS = {
    "cqsa_plan_opts_default": (None, [ctypes.POINTER(cqsa_plan_opts)]),
    "cqsa_plan": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                 ctypes.c_uint64, ctypes.POINTER(cqsa_plan_opts),
                                 ctypes.POINTER(ctypes.c_void_p)]),
    "cqsa_plan_depth": (ctypes.c_int32, [ctypes.c_void_p]),
    "cqsa_plan_num_tasks": (ctypes.c_int64, [ctypes.c_void_p]),
    "cqsa_plan_get_task": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(cqsa_task)]),
    "cqsa_plan_modelled_device_bytes": (ctypes.c_uint64, [ctypes.c_void_p]),
    "cqsa_plan_tasks_per_slot": (ctypes.c_int32, [ctypes.c_void_p]),
    "cqsa_plan_bwd_tasks_per_launch": (ctypes.c_int32, [ctypes.c_void_p]),
    "cqsa_plan_acc_on_device": (ctypes.c_int32, [ctypes.c_void_p]),
    "cqsa_plan_reads_in_place": (ctypes.c_int32, [ctypes.c_void_p]),
    "cqsa_plan_tile_census": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64),
                                             ctypes.POINTER(ctypes.c_int64),
                                             ctypes.POINTER(ctypes.c_int64)]),
    "cqsa_plan_fwd_tile_decisions": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64),
                                                    ctypes.POINTER(ctypes.c_int64),
                                                    ctypes.POINTER(ctypes.c_int64)]),
    "cqsa_bwd_kv_query_tile": (ctypes.c_int32, [ctypes.c_int32]),
    "cqsa_plan_bwd_tile_decisions": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64),
                                                    ctypes.POINTER(ctypes.c_int64)]),
    "cqsa_plan_destroy": (None, [ctypes.c_void_p]),
    "cqsa_forward": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(cqsa_tensor),
                                    ctypes.POINTER(cqsa_tensor), ctypes.POINTER(cqsa_tensor),
                                    ctypes.POINTER(cqsa_tensor), ctypes.c_void_p, ctypes.c_int,
                                    ctypes.c_float, ctypes.c_void_p]),
    "cqsa_forward_noalloc": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(cqsa_tensor),
                                            ctypes.POINTER(cqsa_tensor), ctypes.POINTER(cqsa_tensor),
                                            ctypes.POINTER(cqsa_tensor), ctypes.c_void_p, ctypes.c_int,
                                            ctypes.c_float, ctypes.c_void_p]),
    "cqsa_backward": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(cqsa_tensor),
                                     ctypes.POINTER(cqsa_tensor), ctypes.POINTER(cqsa_tensor),
                                     ctypes.POINTER(cqsa_tensor), ctypes.c_void_p, ctypes.c_int,
                                     ctypes.POINTER(cqsa_tensor), ctypes.POINTER(cqsa_tensor),
                                     ctypes.POINTER(cqsa_tensor), ctypes.POINTER(cqsa_tensor),
                                     ctypes.c_float, ctypes.c_void_p]),
    "cqsa_set_allocator": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "cqsa_set_timing": (ctypes.c_int, [ctypes.c_int32]),
    "cqsa_set_tile_counting": (ctypes.c_int, [ctypes.c_int32]),
    "cqsa_last_stats": (ctypes.c_int, [ctypes.POINTER(cqsa_run_stats)]),
    "cqsa_release_workspace": (ctypes.c_int, []),
    "cqsa_last_error": (ctypes.c_char_p, []),
}

_lib = None


def lib():
    """The loaded native library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2604_20819_amd.build` (no fallback exists)")
        so = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(so, name)
            fn.restype = res
            fn.argtypes = args
        _lib = so
    return _lib


def _check(status, what):
    if status != 0:
        msg = lib().cqsa_last_error().decode(errors="replace")
        raise CqsaError(status, f"{what}: {msg}")


def cqsa_plan_opts_default():
    o = cqsa_plan_opts()
    lib().cqsa_plan_opts_default(ctypes.byref(o))
    return o


def make_opts(B=1, dtype="bf16", c=7, interest=(0, 1, 3), depth=-1, min_depth=1, max_depth=4,
              n_slots=2, inputs_on_device=True, acc_on_device=True, with_backward=False,
              tasks_per_slot=0, levels=None, read_in_place=None, out16=False,
              bwd_tasks_per_launch=0):
    """levels: optional list of (c, interest) per depth (the last repeats below).
    acc_on_device=None asks the planner to choose the accumulator residency;
    read_in_place=None lets it choose whether the kernels read the caller's
    tensors in place (True) or gather each task's runs first (False).
    out16=True makes cqsa_forward write O in the input dtype.
    bwd_tasks_per_launch: 0 automatic, n >= 1 backward tasks per launch."""
    o = cqsa_plan_opts_default()
    o.B = B
    o.dtype = {"f32": CQSA_F32, "f16": CQSA_F16, "bf16": CQSA_BF16}[dtype]
    o.c = c
    o.l = len(interest)
    for i in range(16):
        o.interest[i] = interest[i] if i < len(interest) else 0
    o.depth, o.min_depth, o.max_depth, o.n_slots = depth, min_depth, max_depth, n_slots
    o.inputs_on_device = int(bool(inputs_on_device))
    o.acc_on_device = -1 if acc_on_device is None else int(bool(acc_on_device))
    o.with_backward = int(bool(with_backward))
    o.tasks_per_slot = int(tasks_per_slot)
    o.read_in_place = -1 if read_in_place is None else int(bool(read_in_place))
    o.out16 = int(bool(out16))
    o.bwd_tasks_per_launch = int(bwd_tasks_per_launch)
    if levels:
        if len(levels) > 4:
            raise ValueError("at most 4 level sets")
        o.n_level_sets = len(levels)
        for k, (lc, li) in enumerate(levels):
            o.level_sets[k].c = lc
            o.level_sets[k].l = len(li)
            for i in range(16):
                o.level_sets[k].interest[i] = li[i] if i < len(li) else 0
    return o


class Plan:
    """Owner of a cqsa_plan_t*."""

    def __init__(self, handle, opts, L, H, d, causal):
        self.handle = handle
        self.opts = opts
        self.L, self.H, self.d, self.causal = L, H, d, causal

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.cqsa_plan_destroy(self.handle)
            self.handle = None

    @property
    def depth(self):
        return lib().cqsa_plan_depth(self.handle)

    @property
    def num_tasks(self):
        return lib().cqsa_plan_num_tasks(self.handle)

    @property
    def modelled_device_bytes(self):
        return lib().cqsa_plan_modelled_device_bytes(self.handle)

    @property
    def tasks_per_slot(self):
        return lib().cqsa_plan_tasks_per_slot(self.handle)

    @property
    def bwd_tasks_per_launch(self):
        return lib().cqsa_plan_bwd_tasks_per_launch(self.handle)

    @property
    def acc_on_device(self):
        return lib().cqsa_plan_acc_on_device(self.handle)

    @property
    def reads_in_place(self):
        return lib().cqsa_plan_reads_in_place(self.handle)

    def task(self, t):
        """Task t as a dict of plain Python values."""
        tk = cqsa_task()
        _check(lib().cqsa_plan_get_task(self.handle, t, ctypes.byref(tk)), "cqsa_plan_get_task")
        return dict(index=tk.index, depth=tk.depth,
                    quorum=tuple(tk.quorum[i] for i in range(tk.depth)),
                    L_local=tk.L_local,
                    runs=[(tk.runs[i].global_start, tk.runs[i].length, tk.runs[i].bits)
                          for i in range(tk.n_runs)],
                    block_or=[tk.block_or[i] for i in range(tk.n_blocks)],
                    block_and=[tk.block_and[i] for i in range(tk.n_blocks)])

    def tile_census(self):
        f, c, m = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(lib().cqsa_plan_tile_census(self.handle, ctypes.byref(f), ctypes.byref(c),
                                           ctypes.byref(m)), "cqsa_plan_tile_census")
        return f.value, c.value, m.value

    def fwd_tile_decisions(self):
        """(masked, clear, mixed) the inner forward's tile decisions should
        count (cqsa_plan_fwd_tile_decisions)."""
        f, c, m = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(lib().cqsa_plan_fwd_tile_decisions(self.handle, ctypes.byref(f), ctypes.byref(c),
                                                  ctypes.byref(m)), "cqsa_plan_fwd_tile_decisions")
        return f.value, c.value, m.value

    def bwd_tile_decisions(self):
        """((dQ masked, clear, mixed), (dK/dV masked, clear, mixed)) the
        backward kernels' tile decisions should count
        (cqsa_plan_bwd_tile_decisions)."""
        dq, kv = (ctypes.c_int64 * 3)(), (ctypes.c_int64 * 3)()
        _check(lib().cqsa_plan_bwd_tile_decisions(self.handle, dq, kv), "cqsa_plan_bwd_tile_decisions")
        return tuple(dq), tuple(kv)


def cqsa_bwd_kv_query_tile(d):
    """Query rows of one dK/dV tile at head dim d (cqsa_bwd_kv_query_tile)."""
    return lib().cqsa_bwd_kv_query_tile(d)


def cqsa_plan(L, H, d, causal, device_budget_bytes=0, opts=None):
    """Plan a call (host only).  opts: a cqsa_plan_opts (make_opts) or None."""
    h = ctypes.c_void_p()
    po = ctypes.byref(opts) if opts is not None else None
    _check(lib().cqsa_plan(L, H, d, int(bool(causal)), int(device_budget_bytes), po,
                           ctypes.byref(h)), "cqsa_plan")
    return Plan(h.value, opts if opts is not None else cqsa_plan_opts_default(), L, H, d, causal)


# ---------------------------------------------------------------- torch glue
def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    return {torch.float32: CQSA_F32, torch.float16: CQSA_F16, torch.bfloat16: CQSA_BF16}[t.dtype]


def as_cqsa_tensor(t):
    """Describe a contiguous [B, L, H, d] torch tensor (no copy)."""
    if t.dim() != 4:
        raise ValueError("tensors must be [B, L, H, d]")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return cqsa_tensor(t.data_ptr(), _dtype_code(t),
                       CQSA_MEM_DEVICE if t.is_cuda else CQSA_MEM_HOST, *t.shape)


def _stream_of(*ts):
    torch = _torch()
    for t in ts:
        if t is not None and t.is_cuda:
            return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)
    return ctypes.c_void_p(0)


def _check_lse(plan, LSE, O):
    """The C ABI takes LSE as a bare float pointer: its shape, dtype, layout and
    residency are checked here, before any call."""
    if LSE.dtype != _torch().float32 or not LSE.is_contiguous():
        raise ValueError("LSE must be a contiguous float32 tensor")
    want = (plan.opts.B, plan.H, plan.L)
    if tuple(LSE.shape) != want:
        raise ValueError(f"LSE must have shape (B, H, L) = {want}, got {tuple(LSE.shape)}")
    if LSE.is_cuda != O.is_cuda or (LSE.is_cuda and LSE.device != O.device):
        raise ValueError("LSE must live where O lives")


def cqsa_forward(plan, Q, K, V, O, LSE, scale=0.0, stream=None):
    """O (fp32 [B,L,H,d], or the input dtype with out16) and LSE (fp32 [B,H,L]) are
    written in place."""
    _check_lse(plan, LSE, O)
    tq, tk, tv, to = (as_cqsa_tensor(x) for x in (Q, K, V, O))
    s = stream if stream is not None else _stream_of(O, Q)
    _check(lib().cqsa_forward(plan.handle, ctypes.byref(tq), ctypes.byref(tk), ctypes.byref(tv),
                              ctypes.byref(to), ctypes.c_void_p(LSE.data_ptr()),
                              CQSA_MEM_DEVICE if LSE.is_cuda else CQSA_MEM_HOST,
                              float(scale), s), "cqsa_forward")


def cqsa_forward_noalloc(plan, Q, K, V, O, LSE, scale=0.0, stream=None):
    """cqsa_forward working in the device's fixed scratch array: allocates
    nothing (for graph capture and serving loops); see include/cqsa.h for its
    limits."""
    _check_lse(plan, LSE, O)
    tq, tk, tv, to = (as_cqsa_tensor(x) for x in (Q, K, V, O))
    s = stream if stream is not None else _stream_of(O, Q)
    _check(lib().cqsa_forward_noalloc(plan.handle, ctypes.byref(tq), ctypes.byref(tk),
                                      ctypes.byref(tv), ctypes.byref(to),
                                      ctypes.c_void_p(LSE.data_ptr()),
                                      CQSA_MEM_DEVICE if LSE.is_cuda else CQSA_MEM_HOST,
                                      float(scale), s), "cqsa_forward_noalloc")


def cqsa_backward(plan, Q, K, V, O, LSE, dO, dQ, dK, dV, scale=0.0, stream=None):
    """dQ, dK, dV (fp32 [B,L,H,d]) are overwritten.  Q, K, V, dO live where the
    plan's inputs do; O, LSE, dQ, dK, dV where its accumulator does."""
    _check_lse(plan, LSE, O)
    ts = [as_cqsa_tensor(x) for x in (Q, K, V, O, dO, dQ, dK, dV)]
    s = stream if stream is not None else _stream_of(dQ, Q)
    _check(lib().cqsa_backward(plan.handle, *(ctypes.byref(t) for t in ts[:4]),
                               ctypes.c_void_p(LSE.data_ptr()),
                               CQSA_MEM_DEVICE if LSE.is_cuda else CQSA_MEM_HOST,
                               *(ctypes.byref(t) for t in ts[4:]), float(scale), s),
           "cqsa_backward")


def cqsa_set_timing(enable):
    _check(lib().cqsa_set_timing(int(bool(enable))), "cqsa_set_timing")


def cqsa_set_tile_counting(enable):
    _check(lib().cqsa_set_tile_counting(int(bool(enable))), "cqsa_set_tile_counting")


def cqsa_last_stats():
    st = cqsa_run_stats()
    _check(lib().cqsa_last_stats(ctypes.byref(st)), "cqsa_last_stats")
    return {name: getattr(st, name) for name, _ in cqsa_run_stats._fields_}


def cqsa_release_workspace():
    _check(lib().cqsa_release_workspace(), "cqsa_release_workspace")


_ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p)
_RELEASE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p)
_hooks = None  # the installed callbacks, kept alive while the library may call them


def cqsa_set_allocator(alloc=None, release=None):
    """Route the library's device workspace through alloc(nbytes) -> int device
    address (0 = failure) and release(address); None for both restores the
    built-in cached workspace."""
    global _hooks
    if (alloc is None) != (release is None):
        raise ValueError("give both functions or neither")
    if alloc is None:
        _check(lib().cqsa_set_allocator(None, None, None), "cqsa_set_allocator")
        _hooks = None
        return
    a = _ALLOC_FN(lambda n, ctx: alloc(int(n)) or None)
    r = _RELEASE_FN(lambda ptr, ctx: release(int(ptr)))
    _check(lib().cqsa_set_allocator(ctypes.cast(a, ctypes.c_void_p), ctypes.cast(r, ctypes.c_void_p),
                                    None), "cqsa_set_allocator")
    _hooks = (a, r)


def use_torch_allocator(device=None):
    """Serve the workspace from torch's caching allocator (on `device`)."""
    torch = _torch()
    held = {}

    def alloc(n):
        t = torch.empty((n,), dtype=torch.uint8, device=device or "cuda")
        held[t.data_ptr()] = t
        return t.data_ptr()

    def release(ptr):
        held.pop(ptr, None)

    cqsa_set_allocator(alloc, release)
    return held


def forward(Q, K, V, causal, device_budget_bytes=0, depth=-1, scale=0.0, **opt_kw):
    """Plan and run a forward; returns (O, LSE, plan).  Outputs live where Q lives
    unless acc_on_device is given."""
    torch = _torch()
    B, L, H, d = Q.shape
    dt = {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}[Q.dtype]
    opt_kw.setdefault("inputs_on_device", Q.is_cuda)
    opt_kw.setdefault("acc_on_device", Q.is_cuda)
    opts = make_opts(B=B, dtype=dt, depth=depth, **opt_kw)
    plan = cqsa_plan(L, H, d, causal, device_budget_bytes, opts)
    dev = Q.device if opts.acc_on_device else torch.device("cpu")
    pin = not opts.acc_on_device and torch.cuda.is_available()
    O = torch.empty((B, L, H, d), dtype=torch.float32, device=dev, pin_memory=pin)
    LSE = torch.empty((B, H, L), dtype=torch.float32, device=dev, pin_memory=pin)
    cqsa_forward(plan, Q, K, V, O, LSE, scale)
    return O, LSE, plan
