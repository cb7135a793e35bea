"""Python binding of libhalo_attn.so (ctypes; argument marshalling only).

Every step of the attention path runs in the library's HIP kernels. This
module turns torch tensors into device pointers, numpy arrays into the host
forest, and status codes into exceptions. There is no CPU fallback: without
the built library every call raises.
"""

import ctypes
import os

import numpy as np

from .build import LIB_PATH

HALO_OK = 0
HALO_ERR_INVALID_ARGUMENT = 1
HALO_ERR_UNSUPPORTED = 2
HALO_ERR_WORKSPACE_TOO_SMALL = 3
HALO_ERR_HIP = 4
HALO_ERR_REPLAN = 5

HALO_F32 = 0
HALO_BF16 = 1
HALO_POOL_K = 0
HALO_POOL_V = 1

_I32P = ctypes.POINTER(ctypes.c_int32)


class AttnParams(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_pool_pages", ctypes.c_int64), ("kv_dtype", ctypes.c_int),
                ("out_dtype", ctypes.c_int), ("sm_scale", ctypes.c_float)]


class Forest(ctypes.Structure):
    _fields_ = [("num_segments", ctypes.c_int32), ("seg_len", _I32P),
                ("seg_page_indptr", _I32P), ("seg_page_ids", _I32P),
                ("num_requests", ctypes.c_int32), ("req_seg_indptr", _I32P),
                ("req_seg_ids", _I32P), ("q_len", _I32P)]


class PlanStats(ctypes.Structure):
    _fields_ = [("is_prefill", ctypes.c_int32), ("num_items", ctypes.c_int32),
                ("num_shared_items", ctypes.c_int32), ("num_merge_rows", ctypes.c_int32),
                ("num_partial_rows", ctypes.c_int64), ("num_query_rows", ctypes.c_int64),
                ("distinct_kv_tokens", ctypes.c_int64), ("visible_pairs", ctypes.c_int64),
                ("num_wide_items", ctypes.c_int32), ("wide_row_blocks", ctypes.c_int32)]


class PlanLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in (
        "seg_page_off", "seg_len", "page_ids", "items", "wide_items", "spans", "rows", "merge_rows",
        "merge_indptr", "merge_parts", "total_bytes", "item_recs")] + [(n, ctypes.c_int32) for n in (
            "n_items", "n_wide", "n_spans", "n_rows", "n_merge", "n_merge_parts", "n_pages",
            "n_narrow_blocks", "narrow_slots")]


class PlanOptions(ctypes.Structure):
    """halo_plan_options_t: tuning of the work decomposition (0 / -1 = chosen
    by the planner); see include/halo_attn.h."""
    _fields_ = [(n, ctypes.c_int32) for n in (
        "kc_shared", "kc_private", "wide", "wide_rows", "kc_wide", "wide_min_items", "shared_unit",
        "items_per_block", "append_reserve")]


EXPORTED_SYMBOLS = (
    "halo_plan_create", "halo_plan_create_with_options", "halo_plan_options_default", "halo_plan_upload",
    "halo_plan_upload_update", "halo_plan_destroy", "halo_plan_get_stats", "halo_plan_update_lengths",
    "halo_plan_inspect",
    "halo_prefix_attn_decode", "halo_prefix_attn_prefill", "halo_prefix_attn_decode_noalloc",
    "halo_kv_page_gather",
    "halo_kv_page_scatter", "halo_kv_page_scatter_kv", "halo_kv_page_copy",
    "halo_prefix_tree_build", "halo_prefix_tree_get", "halo_prefix_tree_destroy",
    "halo_status_string", "halo_last_error_message",
)


class PrefixTreeInfo(ctypes.Structure):
    _fields_ = [("num_segments", ctypes.c_int32), ("num_path_entries", ctypes.c_int32),
                ("num_pages", ctypes.c_int64), ("prompt_tokens", ctypes.c_int64),
                ("distinct_tokens", ctypes.c_int64)]


class HaloError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{_status_name(status)}: {message}")
        self.status = status


_LIB = None


def _status_name(status):
    names = {0: "HALO_OK", 1: "HALO_ERR_INVALID_ARGUMENT", 2: "HALO_ERR_UNSUPPORTED",
             3: "HALO_ERR_WORKSPACE_TOO_SMALL", 4: "HALO_ERR_HIP", 5: "HALO_ERR_REPLAN"}
    return names.get(status, f"status {status}")


def _hip_runtimes_mapped():
    try:
        with open("/proc/self/maps") as f:
            paths = {line.split()[-1] for line in f if "libamdhip64" in line}
    except OSError:
        return set()
    return {os.path.realpath(p) for p in paths}


def load_library(require_gpu=False):
    """Load the built library (once). With require_gpu, torch is imported
    first so the process maps a single HIP runtime (torch's), and a GPU must
    be visible."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if require_gpu:
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU visible to torch")
        torch.cuda.init()
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2509_02121_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    lib.halo_plan_create.argtypes = [ctypes.POINTER(AttnParams), ctypes.POINTER(Forest),
                                     ctypes.POINTER(vp), ctypes.POINTER(sz), ctypes.POINTER(sz)]
    lib.halo_plan_create.restype = ctypes.c_int
    lib.halo_plan_create_with_options.argtypes = [ctypes.POINTER(AttnParams), ctypes.POINTER(Forest),
                                                  ctypes.POINTER(PlanOptions), ctypes.POINTER(vp),
                                                  ctypes.POINTER(sz), ctypes.POINTER(sz)]
    lib.halo_plan_create_with_options.restype = ctypes.c_int
    lib.halo_plan_options_default.argtypes = [ctypes.POINTER(PlanOptions)]
    lib.halo_plan_options_default.restype = None
    lib.halo_plan_update_lengths.argtypes = [vp, ctypes.POINTER(Forest)]
    lib.halo_plan_update_lengths.restype = ctypes.c_int
    lib.halo_plan_upload.argtypes = [vp, vp, sz, vp]
    lib.halo_plan_upload.restype = ctypes.c_int
    lib.halo_plan_upload_update.argtypes = [vp, vp, sz, vp]
    lib.halo_plan_upload_update.restype = ctypes.c_int
    lib.halo_plan_destroy.argtypes = [vp]
    lib.halo_plan_destroy.restype = None
    lib.halo_plan_get_stats.argtypes = [vp, ctypes.POINTER(PlanStats)]
    lib.halo_plan_get_stats.restype = ctypes.c_int
    lib.halo_plan_inspect.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(PlanLayout)]
    lib.halo_plan_inspect.restype = ctypes.c_int
    for name in ("halo_prefix_attn_decode", "halo_prefix_attn_prefill"):
        fn = getattr(lib, name)
        fn.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        fn.restype = ctypes.c_int
    lib.halo_prefix_attn_decode_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp]
    lib.halo_prefix_attn_decode_noalloc.restype = ctypes.c_int
    lib.halo_kv_page_gather.argtypes = [vp, ctypes.POINTER(AttnParams), ctypes.c_int, vp, vp, vp, vp,
                                        ctypes.c_int32, vp, vp, vp]
    lib.halo_kv_page_gather.restype = ctypes.c_int
    lib.halo_kv_page_scatter.argtypes = [vp, ctypes.POINTER(AttnParams), ctypes.c_int, vp, vp, vp, vp, vp,
                                         ctypes.c_int32, vp, vp, vp]
    lib.halo_kv_page_scatter.restype = ctypes.c_int
    lib.halo_kv_page_scatter_kv.argtypes = [vp, vp, ctypes.POINTER(AttnParams), vp, vp, vp, vp, vp,
                                            ctypes.c_int32, vp, vp, vp, vp]
    lib.halo_kv_page_scatter_kv.restype = ctypes.c_int
    lib.halo_kv_page_copy.argtypes = [vp, ctypes.POINTER(AttnParams), vp, vp, ctypes.c_int32, vp, vp]
    lib.halo_kv_page_copy.restype = ctypes.c_int
    lib.halo_prefix_tree_build.argtypes = [vp, vp, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(vp),
                                           ctypes.POINTER(PrefixTreeInfo)]
    lib.halo_prefix_tree_build.restype = ctypes.c_int
    lib.halo_prefix_tree_get.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp]
    lib.halo_prefix_tree_get.restype = ctypes.c_int
    lib.halo_prefix_tree_destroy.argtypes = [vp]
    lib.halo_prefix_tree_destroy.restype = None
    lib.halo_status_string.argtypes = [ctypes.c_int]
    lib.halo_status_string.restype = ctypes.c_char_p
    lib.halo_last_error_message.argtypes = []
    lib.halo_last_error_message.restype = ctypes.c_char_p
    if require_gpu:
        runtimes = _hip_runtimes_mapped()
        if len(runtimes) > 1:
            raise RuntimeError(f"several HIP runtimes mapped: {sorted(runtimes)}")
    _LIB = lib
    return lib


def _check(status):
    if status != HALO_OK:
        msg = _LIB.halo_last_error_message().decode()
        raise HaloError(status, msg)


def _dtype_code(dtype):
    import torch
    if dtype == torch.float32:
        return HALO_F32
    if dtype == torch.bfloat16:
        return HALO_BF16
    raise ValueError(f"unsupported dtype {dtype}")


def _torch_dtype(code):
    import torch
    return {HALO_F32: torch.float32, HALO_BF16: torch.bfloat16}[code]


def _gpu(t, name, dtype=None, min_numel=None):
    """Check that t is a contiguous GPU tensor (of dtype, with at least
    min_numel elements): the C ABI takes raw pointers, so a strided view, a
    host tensor or another element type would be read as garbage."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs at least {min_numel}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    return t


def _page_lists(page_ids, seq_page_indptr):
    """Check the int32 page lists; returns the number of sequences."""
    import torch
    _gpu(seq_page_indptr, "seq_page_indptr", torch.int32, 1)
    _gpu(page_ids, "page_ids", torch.int32)
    return int(seq_page_indptr.numel() - 1)


def make_params(num_q_heads, num_kv_heads, head_dim, kv_dtype, num_pool_pages, sm_scale,
                out_dtype=None, page_size=16):
    """AttnParams from Python values (dtypes as torch dtypes)."""
    return AttnParams(num_q_heads, num_kv_heads, head_dim, page_size, int(num_pool_pages),
                      _dtype_code(kv_dtype), _dtype_code(out_dtype if out_dtype is not None else kv_dtype),
                      float(sm_scale))


def _i32(a):
    return None if a is None else np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_I32P)


class Plan:
    """A validated forest plus the work lists of one batch step (host)."""

    def __init__(self, params, seg_len, seg_page_indptr, seg_page_ids, req_seg_indptr,
                 req_seg_ids, q_len=None, options=None):
        """options: None (the planner's choices) or a dict of
        halo_plan_options_t fields to set."""
        lib = load_library()
        self.params = params
        keep = [_i32(x) for x in (seg_len, seg_page_indptr, seg_page_ids, req_seg_indptr,
                                  req_seg_ids, q_len)]
        seg_len_a, indptr_a, ids_a, rindptr_a, rids_a, qlen_a = keep
        forest = Forest(len(seg_len_a), _ptr(seg_len_a), _ptr(indptr_a), _ptr(ids_a),
                        len(rindptr_a) - 1, _ptr(rindptr_a), _ptr(rids_a), _ptr(qlen_a))
        handle = ctypes.c_void_p()
        meta = ctypes.c_size_t()
        ws = ctypes.c_size_t()
        self._handle = None
        opts = None
        if options:
            opts = PlanOptions()
            lib.halo_plan_options_default(ctypes.byref(opts))
            for k, v in options.items():
                if k not in dict(PlanOptions._fields_):
                    raise ValueError(f"unknown plan option {k}")
                setattr(opts, k, int(v))
        _check(lib.halo_plan_create_with_options(ctypes.byref(params), ctypes.byref(forest),
                                                 ctypes.byref(opts) if opts is not None else None,
                                                 ctypes.byref(handle), ctypes.byref(meta), ctypes.byref(ws)))
        self._handle = handle
        self._keep = keep
        self.device_meta_bytes = meta.value
        self.workspace_bytes = ws.value
        self.is_prefill = q_len is not None
        self.num_query_rows = int(self.stats()["num_query_rows"])

    @classmethod
    def from_csr(cls, params, csr, options=None):
        return cls(params, csr["seg_len"], csr["seg_page_indptr"], csr["seg_page_ids"],
                   csr["req_seg_indptr"], csr["req_seg_ids"], csr.get("q_len"), options)

    def update_lengths(self, csr):
        """halo_plan_update_lengths with the forest `csr`: True if the plan
        now describes it (re-upload before the next run), False if it
        changed beyond tokens appended inside existing pages (the plan is
        unchanged; build a new one)."""
        keep = [_i32(csr[k]) if csr.get(k) is not None else None
                for k in ("seg_len", "seg_page_indptr", "seg_page_ids", "req_seg_indptr", "req_seg_ids", "q_len")]
        seg_len_a, indptr_a, ids_a, rindptr_a, rids_a, qlen_a = keep
        forest = Forest(len(seg_len_a), _ptr(seg_len_a), _ptr(indptr_a), _ptr(ids_a),
                        len(rindptr_a) - 1, _ptr(rindptr_a), _ptr(rids_a), _ptr(qlen_a))
        st = _LIB.halo_plan_update_lengths(self._handle, ctypes.byref(forest))
        if st == HALO_ERR_REPLAN:
            return False
        _check(st)
        self._keep = keep
        return True

    def image(self):
        """The host metadata image as bytes (a copy)."""
        img = ctypes.c_void_p()
        lay = PlanLayout()
        _check(_LIB.halo_plan_inspect(self._handle, ctypes.byref(img), ctypes.byref(lay)))
        return ctypes.string_at(img.value, lay.total_bytes)

    def stats(self):
        st = PlanStats()
        _check(_LIB.halo_plan_get_stats(self._handle, ctypes.byref(st)))
        return {f: getattr(st, f) for f, _ in PlanStats._fields_}

    def inspect(self):
        """The host metadata image decoded into numpy arrays (a copy)."""
        img = ctypes.c_void_p()
        lay = PlanLayout()
        _check(_LIB.halo_plan_inspect(self._handle, ctypes.byref(img), ctypes.byref(lay)))
        raw = np.frombuffer(ctypes.string_at(img.value, lay.total_bytes), dtype=np.uint8)

        def arr(off, count, width=1):
            a = raw[off:off + 4 * count * width].view(np.int32)
            return a.reshape(count, width) if width > 1 else a.copy()

        S = len(self._keep[0])
        return dict(
            seg_page_off=arr(lay.seg_page_off, S), seg_len=arr(lay.seg_len, S),
            page_ids=arr(lay.page_ids, lay.n_pages),
            items=arr(lay.items, lay.n_items, 16).copy(),
            item_recs=arr(lay.item_recs, lay.n_items, 64).copy(),
            n_narrow_blocks=lay.n_narrow_blocks, narrow_slots=lay.narrow_slots,
            wide_items=arr(lay.wide_items, lay.n_wide, 16).copy(), spans=arr(lay.spans, lay.n_spans, 8).copy(),
            rows=arr(lay.rows, lay.n_rows, 4).copy(), merge_rows=arr(lay.merge_rows, lay.n_merge),
            merge_indptr=arr(lay.merge_indptr, lay.n_merge + 1),
            merge_parts=arr(lay.merge_parts, lay.n_merge_parts), total_bytes=lay.total_bytes)

    def upload(self, device_meta, stream=None):
        _check(_LIB.halo_plan_upload(self._handle, device_meta.data_ptr(),
                                     device_meta.numel() * device_meta.element_size(),
                                     _stream_handle(stream)))

    def upload_update(self, device_meta, stream=None):
        """halo_plan_upload_update: only what update_lengths changes, into a
        buffer that already holds an upload of this plan."""
        _check(_LIB.halo_plan_upload_update(self._handle, device_meta.data_ptr(),
                                            device_meta.numel() * device_meta.element_size(),
                                            _stream_handle(stream)))

    def close(self):
        if self._handle is not None and _LIB is not None:
            _LIB.halo_plan_destroy(self._handle)
        self._handle = None

    def __del__(self):
        self.close()


class PrefixTree:
    """halo_prefix_tree_build on a list of token-id prompts (host only).

    Attributes (numpy int32): seg_len, seg_parent, seg_refcount,
    seg_src_request, seg_src_offset, req_seg_indptr, req_seg_ids; ints
    num_pages, prompt_tokens, distinct_tokens. forest_csr(page_ids) gives the
    forest in the form Plan.from_csr takes."""

    def __init__(self, prompts, page_size=16):
        lib = load_library()
        prompts = [np.asarray(p, dtype=np.int32).ravel() for p in prompts]
        indptr = np.zeros(len(prompts) + 1, dtype=np.int32)
        indptr[1:] = np.cumsum([len(p) for p in prompts])
        tokens = np.ascontiguousarray(np.concatenate(prompts) if prompts else np.zeros(0, np.int32),
                                      dtype=np.int32)
        handle = ctypes.c_void_p()
        info = PrefixTreeInfo()
        _check(lib.halo_prefix_tree_build(_ptr(indptr), _ptr(tokens) if tokens.size else None,
                                          len(prompts), int(page_size), ctypes.byref(handle), ctypes.byref(info)))
        try:
            S, P, R = info.num_segments, info.num_path_entries, len(prompts)
            out = {n: np.zeros(S, np.int32) for n in ("seg_len", "seg_parent", "seg_refcount",
                                                      "seg_src_request", "seg_src_offset")}
            out["req_seg_indptr"] = np.zeros(R + 1, np.int32)
            out["req_seg_ids"] = np.zeros(P, np.int32)
            names = ("seg_len", "seg_parent", "seg_refcount", "seg_src_request", "seg_src_offset",
                     "req_seg_indptr", "req_seg_ids")
            _check(lib.halo_prefix_tree_get(handle, *[_ptr(out[n]) for n in names]))
        finally:
            lib.halo_prefix_tree_destroy(handle)
        for n, a in out.items():
            setattr(self, n, a)
        self.page_size = int(page_size)
        self.num_pages = int(info.num_pages)
        self.prompt_tokens = int(info.prompt_tokens)
        self.distinct_tokens = int(info.distinct_tokens)

    @property
    def num_segments(self):
        return len(self.seg_len)

    def paths(self):
        return [self.req_seg_ids[self.req_seg_indptr[r]:self.req_seg_indptr[r + 1]].tolist()
                for r in range(len(self.req_seg_indptr) - 1)]

    def pages_per_segment(self):
        return (self.seg_len + self.page_size - 1) // self.page_size

    def forest_csr(self, seg_page_ids, q_len=None):
        """The forest with the caller's page ids (seg_page_ids lists, segment
        after segment, pages_per_segment() ids each)."""
        indptr = np.zeros(self.num_segments + 1, dtype=np.int32)
        indptr[1:] = np.cumsum(self.pages_per_segment())
        ids = np.asarray(seg_page_ids, dtype=np.int32)
        if ids.size != indptr[-1]:
            raise ValueError(f"{indptr[-1]} page ids needed, got {ids.size}")
        return dict(seg_len=self.seg_len.copy(), seg_page_indptr=indptr, seg_page_ids=ids,
                    req_seg_indptr=self.req_seg_indptr.copy(), req_seg_ids=self.req_seg_ids.copy(),
                    q_len=None if q_len is None else np.asarray(q_len, np.int32))


def _stream_handle(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _pool_elems(params):
    """Elements of one page pool: num_pool_pages x H_kv x page_size x d."""
    return int(params.num_pool_pages) * params.num_kv_heads * params.page_size * params.head_dim


def _nbytes(t):
    return t.numel() * t.element_size()


def _check_run(plan, device_meta, q, k_pool, v_pool, o, lse, workspace, library_workspace=False):
    """Every buffer a run call reads or writes is checked against the plan's
    sizes before any launch: the kernels index q, o and lse by the plan's
    query rows and the pools by its page ids, so an undersized tensor would
    be read or written out of bounds. Sizes are checked first, then layout,
    element type and device."""
    import torch
    p = plan.params
    kv = _torch_dtype(p.kv_dtype)
    rows = plan.num_query_rows * p.num_q_heads
    need = [(device_meta, "device_meta", plan.device_meta_bytes, "bytes"),
            (k_pool, "k_pool", _pool_elems(p), "elements"), (v_pool, "v_pool", _pool_elems(p), "elements"),
            (o, "o", rows * p.head_dim, "elements")]
    if lse is not None:
        need.append((lse, "lse", rows, "elements"))
    if q.numel() != rows * p.head_dim:
        raise ValueError(f"q has {q.numel()} elements, the plan has {plan.num_query_rows} query rows x "
                         f"{p.num_q_heads} heads x {p.head_dim} = {rows * p.head_dim}")
    for t, name, n, unit in need:
        have = _nbytes(t) if unit == "bytes" else t.numel()
        if have < n:
            raise ValueError(f"{name} has {have} {unit}, the plan needs at least {n}")
    ws = _nbytes(workspace) if workspace is not None else 0
    if not library_workspace and ws < plan.workspace_bytes:
        raise ValueError(f"workspace has {ws} bytes, the plan needs {plan.workspace_bytes}")
    _gpu(device_meta, "device_meta")
    _gpu(q, "q", kv)
    _gpu(k_pool, "k_pool", kv)
    _gpu(v_pool, "v_pool", kv)
    _gpu(o, "o", _torch_dtype(p.out_dtype))
    if lse is not None:
        _gpu(lse, "lse", torch.float32)
    if workspace is not None:
        _gpu(workspace, "workspace")


def _run(fn, plan, device_meta, q, k_pool, v_pool, o, lse, workspace, stream):
    _check_run(plan, device_meta, q, k_pool, v_pool, o, lse, workspace)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(fn(plan._handle, device_meta.data_ptr(), q.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(),
              o.data_ptr(), lse.data_ptr() if lse is not None else None, ws_ptr, ws_bytes,
              _stream_handle(stream)))


def prefix_attn_decode(plan, device_meta, q, k_pool, v_pool, o, lse, workspace, stream=None):
    """halo_prefix_attn_decode on torch tensors (all on one GPU)."""
    _run(_LIB.halo_prefix_attn_decode, plan, device_meta, q, k_pool, v_pool, o, lse, workspace, stream)


def prefix_attn_prefill(plan, device_meta, q, k_pool, v_pool, o, lse, workspace, stream=None):
    """halo_prefix_attn_prefill on torch tensors (all on one GPU)."""
    _run(_LIB.halo_prefix_attn_prefill, plan, device_meta, q, k_pool, v_pool, o, lse, workspace, stream)


# Largest workspace the no-alloc decode entry point serves (HALO_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 64 << 20


def prefix_attn_decode_noalloc(plan, device_meta, q, k_pool, v_pool, o, lse, stream=None):
    """halo_prefix_attn_decode_noalloc on torch tensors: decode with the
    library's own per-GPU scratch instead of a workspace (no allocation).
    Calls that overlap in time on one GPU share that scratch and race."""
    if plan.workspace_bytes > NOALLOC_SCRATCH_BYTES:
        raise ValueError(f"the plan needs {plan.workspace_bytes} bytes of workspace; the no-alloc entry "
                         f"point holds {NOALLOC_SCRATCH_BYTES}")
    _check_run(plan, device_meta, q, k_pool, v_pool, o, lse, None, library_workspace=True)
    _check(_LIB.halo_prefix_attn_decode_noalloc(plan._handle, device_meta.data_ptr(), q.data_ptr(),
                                                k_pool.data_ptr(), v_pool.data_ptr(), o.data_ptr(),
                                                lse.data_ptr() if lse is not None else None,
                                                _stream_handle(stream)))


def _check_gather(pool, params, page_ids, seq_page_indptr, seq_len, out_token_offset, out, error_flag):
    import torch
    kv = _torch_dtype(params.kv_dtype)
    _gpu(pool, "pool", kv, _pool_elems(params))
    n = _page_lists(page_ids, seq_page_indptr)
    _gpu(seq_len, "seq_len", torch.int32, n)
    _gpu(out_token_offset, "out_token_offset", torch.int64, n)
    _gpu(out, "out", kv)
    if error_flag is not None:
        _gpu(error_flag, "error_flag", torch.int32, 1)


def _check_scatter(pools, params, page_ids, seq_page_indptr, seq_start, seq_count, in_token_offset, srcs,
                   error_flag):
    import torch
    kv = _torch_dtype(params.kv_dtype)
    for i, t in enumerate(pools):
        if t.numel() < _pool_elems(params):
            raise ValueError(f"pool {i} has {t.numel()} elements, needs at least {_pool_elems(params)}")
    for i, t in enumerate(pools):
        _gpu(t, f"pool {i}", kv)
    n = _page_lists(page_ids, seq_page_indptr)
    for i, t in enumerate(srcs):
        _gpu(t, f"input {i}", kv)
    _gpu(seq_start, "seq_start", torch.int32, n)
    _gpu(seq_count, "seq_count", torch.int32, n)
    _gpu(in_token_offset, "in_token_offset", torch.int64, n)
    if error_flag is not None:
        _gpu(error_flag, "error_flag", torch.int32, 1)


def _check_copy(pool, params, src_pages, dst_pages, error_flag):
    import torch
    _gpu(pool, "pool", _torch_dtype(params.kv_dtype), _pool_elems(params))
    _gpu(src_pages, "src_pages", torch.int32)
    _gpu(dst_pages, "dst_pages", torch.int32, src_pages.numel())
    if error_flag is not None:
        _gpu(error_flag, "error_flag", torch.int32, 1)


def kv_page_gather(pool, params, pool_kind, page_ids, seq_page_indptr, seq_len, out_token_offset,
                   out, error_flag=None, stream=None):
    """halo_kv_page_gather on torch tensors (int arrays on the GPU)."""
    load_library()
    _check_gather(pool, params, page_ids, seq_page_indptr, seq_len, out_token_offset, out, error_flag)
    _check(_LIB.halo_kv_page_gather(pool.data_ptr(), ctypes.byref(params), int(pool_kind),
                                    page_ids.data_ptr(), seq_page_indptr.data_ptr(), seq_len.data_ptr(),
                                    out_token_offset.data_ptr(), int(seq_page_indptr.numel() - 1),
                                    out.data_ptr(),
                                    error_flag.data_ptr() if error_flag is not None else None,
                                    _stream_handle(stream)))


def kv_page_scatter(pool, params, pool_kind, page_ids, seq_page_indptr, seq_start, seq_count,
                    in_token_offset, src, error_flag=None, stream=None):
    """halo_kv_page_scatter on torch tensors (int arrays on the GPU)."""
    load_library()
    _check_scatter([pool], params, page_ids, seq_page_indptr, seq_start, seq_count, in_token_offset, [src],
                   error_flag)
    _check(_LIB.halo_kv_page_scatter(pool.data_ptr(), ctypes.byref(params), int(pool_kind),
                                     page_ids.data_ptr(), seq_page_indptr.data_ptr(), seq_start.data_ptr(),
                                     seq_count.data_ptr(), in_token_offset.data_ptr(),
                                     int(seq_page_indptr.numel() - 1), src.data_ptr(),
                                     error_flag.data_ptr() if error_flag is not None else None,
                                     _stream_handle(stream)))


def _scatter_kv_args(k_pool, v_pool, params, page_ids, seq_page_indptr, seq_start, seq_count, in_token_offset,
                     k_src, v_src, error_flag, stream):
    _check_scatter([k_pool, v_pool], params, page_ids, seq_page_indptr, seq_start, seq_count, in_token_offset,
                   [k_src, v_src], error_flag)
    return (k_pool.data_ptr(), v_pool.data_ptr(), ctypes.byref(params), page_ids.data_ptr(),
            seq_page_indptr.data_ptr(), seq_start.data_ptr(), seq_count.data_ptr(), in_token_offset.data_ptr(),
            int(seq_page_indptr.numel() - 1), k_src.data_ptr(), v_src.data_ptr(),
            error_flag.data_ptr() if error_flag is not None else None, _stream_handle(stream))


def kv_page_scatter_kv(k_pool, v_pool, params, page_ids, seq_page_indptr, seq_start, seq_count,
                       in_token_offset, k_src, v_src, error_flag=None, stream=None):
    """halo_kv_page_scatter_kv (both pools, one launch) on torch tensors."""
    load_library()
    _check(_LIB.halo_kv_page_scatter_kv(*_scatter_kv_args(k_pool, v_pool, params, page_ids, seq_page_indptr,
                                                          seq_start, seq_count, in_token_offset, k_src, v_src,
                                                          error_flag, stream)))


def kv_page_copy(pool, params, src_pages, dst_pages, error_flag=None, stream=None):
    """halo_kv_page_copy on torch tensors (int arrays on the GPU)."""
    load_library()
    _check_copy(pool, params, src_pages, dst_pages, error_flag)
    _check(_LIB.halo_kv_page_copy(pool.data_ptr(), ctypes.byref(params), src_pages.data_ptr(),
                                  dst_pages.data_ptr(), int(src_pages.numel()),
                                  error_flag.data_ptr() if error_flag is not None else None,
                                  _stream_handle(stream)))


def bind_kv_page_gather(pool, params, pool_kind, page_ids, seq_page_indptr, seq_len, out_token_offset, out,
                        error_flag=None, stream=None):
    """kv_page_gather as a zero-argument callable (see bind_kv_page_scatter)."""
    load_library()
    _check_gather(pool, params, page_ids, seq_page_indptr, seq_len, out_token_offset, out, error_flag)
    args = (pool.data_ptr(), ctypes.byref(params), int(pool_kind), page_ids.data_ptr(), seq_page_indptr.data_ptr(),
            seq_len.data_ptr(), out_token_offset.data_ptr(), int(seq_page_indptr.numel() - 1), out.data_ptr(),
            error_flag.data_ptr() if error_flag is not None else None, _stream_handle(stream))
    fn = _LIB.halo_kv_page_gather

    def call():
        st = fn(*args)
        if st != HALO_OK:
            _check(st)
    return call


def bind_kv_page_scatter(pool, params, pool_kind, page_ids, seq_page_indptr, seq_start, seq_count,
                         in_token_offset, src, error_flag=None, stream=None):
    """A zero-argument callable that enqueues kv_page_scatter with every
    pointer converted once (for tight timing loops); the tensors and params
    must stay alive while it is used."""
    load_library()
    _check_scatter([pool], params, page_ids, seq_page_indptr, seq_start, seq_count, in_token_offset, [src],
                   error_flag)
    args = (pool.data_ptr(), ctypes.byref(params), int(pool_kind), page_ids.data_ptr(),
            seq_page_indptr.data_ptr(), seq_start.data_ptr(), seq_count.data_ptr(),
            in_token_offset.data_ptr(), int(seq_page_indptr.numel() - 1), src.data_ptr(),
            error_flag.data_ptr() if error_flag is not None else None, _stream_handle(stream))
    fn = _LIB.halo_kv_page_scatter

    def call():
        st = fn(*args)
        if st != HALO_OK:
            _check(st)
    return call


def bind_kv_page_scatter_kv(k_pool, v_pool, params, page_ids, seq_page_indptr, seq_start, seq_count,
                            in_token_offset, k_src, v_src, error_flag=None, stream=None):
    """kv_page_scatter_kv as a zero-argument callable (see bind_kv_page_scatter)."""
    load_library()
    args = _scatter_kv_args(k_pool, v_pool, params, page_ids, seq_page_indptr, seq_start, seq_count,
                            in_token_offset, k_src, v_src, error_flag, stream)
    fn = _LIB.halo_kv_page_scatter_kv

    def call():
        st = fn(*args)
        if st != HALO_OK:
            _check(st)
    return call


def bind_kv_page_copy(pool, params, src_pages, dst_pages, error_flag=None, stream=None):
    """kv_page_copy as a zero-argument callable (see bind_kv_page_scatter)."""
    load_library()
    _check_copy(pool, params, src_pages, dst_pages, error_flag)
    args = (pool.data_ptr(), ctypes.byref(params), src_pages.data_ptr(), dst_pages.data_ptr(),
            int(src_pages.numel()), error_flag.data_ptr() if error_flag is not None else None,
            _stream_handle(stream))
    fn = _LIB.halo_kv_page_copy

    def call():
        st = fn(*args)
        if st != HALO_OK:
            _check(st)
    return call


class PrefixAttention:
    """Plan + uploaded metadata + workspace for one forest on one GPU.

    run() enqueues the whole path (attention items, then the merge) on the
    current stream and returns (o, lse).

    The device metadata is double-buffered. update() uploads the next batch
    step's plan into the buffer the current step does not use, on a copy
    stream of its own (or the stream given), after every run already
    enqueued that read that buffer; a run waits for its buffer's upload. The
    copy of step t + 1's plan therefore overlaps step t's kernels, and after
    an in-place update it copies only what the update can change.
    """

    def __init__(self, params, csr, device="cuda", options=None):
        import torch
        load_library(require_gpu=True)
        self.plan = Plan.from_csr(params, csr, options)
        self.options = options
        self.device = torch.device(device)
        self._metas = [self._meta_buffer(self.plan.device_meta_bytes), None]
        self._cur = 0
        self.workspace = (torch.empty(self.plan.workspace_bytes, dtype=torch.uint8, device=self.device)
                          if self.plan.workspace_bytes else None)
        self._copy_stream = torch.cuda.Stream(device=self.device)
        # runs that read buffer i since its last upload: an event after the
        # last run() per stream, and the streams of bound callables (whose
        # calls are not tracked one by one: the upload waits for everything
        # enqueued on those streams)
        self._runs = [{}, {}]
        self._bound = [set(), set()]
        self._uploaded = [None, None]
        self._upload_streams = [None, None]
        # the Plan object whose upload buffer i holds (an in-place update
        # then needs only halo_plan_upload_update)
        self._holds = [None, None]
        self._upload(0, torch.cuda.current_stream(self.device))
        self.out_dtype = {HALO_F32: torch.float32, HALO_BF16: torch.bfloat16}[params.out_dtype]

    @property
    def meta(self):
        """The device metadata buffer of the current plan."""
        return self._metas[self._cur]

    def _meta_buffer(self, nbytes):
        import torch
        return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)

    def _upload(self, i, stream):
        import torch
        for u, ev in self._runs[i].items():
            if u != stream:
                stream.wait_event(ev)
        for u in self._bound[i]:
            if u != stream:
                stream.wait_stream(u)
        self._runs[i].clear()
        self._bound[i].clear()
        if self._holds[i] is self.plan:
            self.plan.upload_update(self._metas[i], stream)
        else:
            self.plan.upload(self._metas[i], stream)
            self._holds[i] = self.plan
        ev = torch.cuda.Event()
        ev.record(stream)
        self._uploaded[i] = ev
        self._upload_streams[i] = stream

    def update(self, csr, stream=None):
        """Bring the plan up to date with `csr` (the next decode step's
        forest): the length update when it applies, else a new plan (with
        larger metadata and workspace buffers if needed). Uploads the new
        metadata into the other buffer, on `stream` (None: this object's copy
        stream). Callables from bind() keep the plan they were bound with:
        bind again after update(). Returns True if the update applied."""
        import torch
        # the last upload read the host image asynchronously
        self._uploaded[self._cur].synchronize()
        applied = self.plan.update_lengths(csr)
        nxt = 1 - self._cur
        if not applied:
            self.plan = Plan.from_csr(self.plan.params, csr, self.options)
            ws_have = self.workspace.numel() if self.workspace is not None else 0
            if self.plan.workspace_bytes > ws_have:
                # runs in flight may still use the old workspace
                torch.cuda.synchronize(self.device)
                self.workspace = torch.empty(self.plan.workspace_bytes, dtype=torch.uint8, device=self.device)
        if self._metas[nxt] is None or self._metas[nxt].numel() < self.plan.device_meta_bytes:
            torch.cuda.synchronize(self.device)
            self._metas[nxt] = self._meta_buffer(self.plan.device_meta_bytes)
            self._holds[nxt] = None
        self._upload(nxt, stream if stream is not None else self._copy_stream)
        self._cur = nxt
        return applied

    def _before_run(self, stream):
        """Make `stream` (None: the current stream) wait for the current
        buffer's upload; returns that stream."""
        import torch
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        if s != self._upload_streams[self._cur]:
            s.wait_event(self._uploaded[self._cur])
        return s

    def _after_run(self, s):
        """Note that the run just enqueued on `s` reads the current buffer."""
        import torch
        ev = torch.cuda.Event()
        ev.record(s)
        self._runs[self._cur][s] = ev

    def alloc_outputs(self, q):
        import torch
        o = torch.empty(q.shape, dtype=self.out_dtype, device=q.device)
        lse = torch.empty(q.shape[:2], dtype=torch.float32, device=q.device)
        return o, lse

    def bind(self, q, k_pool, v_pool, o, lse, stream=None):
        """A zero-argument callable that enqueues run(q, k_pool, v_pool, o,
        lse) with every pointer converted once (for tight timing loops).
        The tensors must stay alive while the callable is used."""
        fn = _LIB.halo_prefix_attn_prefill if self.plan.is_prefill else _LIB.halo_prefix_attn_decode
        ws = self.workspace
        _check_run(self.plan, self.meta, q, k_pool, v_pool, o, lse, ws)
        self._bound[self._cur].add(self._before_run(stream))
        args = (self.plan._handle, self.meta.data_ptr(), q.data_ptr(), k_pool.data_ptr(),
                v_pool.data_ptr(), o.data_ptr(), lse.data_ptr() if lse is not None else None,
                ws.data_ptr() if ws is not None else None,
                ws.numel() if ws is not None else 0, _stream_handle(stream))

        def call():
            st = fn(*args)
            if st != HALO_OK:
                _check(st)
        return call

    def run(self, q, k_pool, v_pool, o=None, lse=None, stream=None):
        if o is None:
            o, lse_new = self.alloc_outputs(q)
            lse = lse if lse is not None else lse_new
        fn = prefix_attn_prefill if self.plan.is_prefill else prefix_attn_decode
        s = self._before_run(stream)
        fn(self.plan, self.meta, q, k_pool, v_pool, o, lse, self.workspace, stream)
        self._after_run(s)
        return o, lse
