"""Thin ctypes binding over ``libnuna.so`` (C ABI in ``include/nuna.h``).

Argument marshalling only: every collective runs in the library's gfx950
kernels.  Torch tensors supply device memory and the stream; nothing here
computes on the host, and there is no fallback: if the library is missing,
loading it raises.

Two layers:

* ``raw`` functions take integer device pointers and return the status code
  (used to exercise the C ABI directly, including its argument checks);
* tensor functions take lists of CUDA tensors (one per simulated rank),
  enqueue on the current torch stream and raise ``NunaError`` on failure.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnuna.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_MISALIGNED, ERR_OVERLAP, ERR_HIP, ERR_NO_MEMORY = range(7)
STATUS_NAMES = {0: "NUNA_OK", 1: "NUNA_ERR_INVALID_ARG", 2: "NUNA_ERR_UNSUPPORTED", 3: "NUNA_ERR_MISALIGNED",
                4: "NUNA_ERR_OVERLAP", 5: "NUNA_ERR_HIP", 6: "NUNA_ERR_NO_MEMORY"}
F32, BF16 = 0, 1
LINEAR, XCD = 0, 1
ALGO_AUTO, ALGO_ONE_SHOT, ALGO_TWO_SHOT, ALGO_ONE_SHOT_SPLIT, ALGO_TWO_SHOT_TWO_KERNELS = 0, 1, 2, 3, 4

PLACEMENTS = {"linear": LINEAR, "xcd": XCD, LINEAR: LINEAR, XCD: XCD}
ALGOS = {"auto": ALGO_AUTO, "one_shot": ALGO_ONE_SHOT, "two_shot": ALGO_TWO_SHOT, "one_shot_split": ALGO_ONE_SHOT_SPLIT,
         "two_shot_two_kernels": ALGO_TWO_SHOT_TWO_KERNELS,
         ALGO_AUTO: ALGO_AUTO, ALGO_ONE_SHOT: ALGO_ONE_SHOT, ALGO_TWO_SHOT: ALGO_TWO_SHOT,
         ALGO_ONE_SHOT_SPLIT: ALGO_ONE_SHOT_SPLIT, ALGO_TWO_SHOT_TWO_KERNELS: ALGO_TWO_SHOT_TWO_KERNELS}

_vp = ctypes.c_void_p
_vpp = ctypes.POINTER(ctypes.c_void_p)
_i64p = ctypes.POINTER(ctypes.c_int64)
_i32p = ctypes.POINTER(ctypes.c_int32)

NAP_MAX_DOMAINS = 16
NAP_MAX_STACKS = 16


class DeviceInfo(ctypes.Structure):
    """Mirror of nuna_device_info_t."""
    _fields_ = [("device", ctypes.c_int32), ("cu_count", ctypes.c_int32), ("xcd_count", ctypes.c_int32),
                ("map_verified", ctypes.c_int32)]


class LaunchInfo(ctypes.Structure):
    """Mirror of nuna_launch_info_t."""
    _fields_ = [("kernels", ctypes.c_char * 96), ("launches", ctypes.c_int32), ("map", ctypes.c_int32),
                ("group_size", ctypes.c_int64), ("grid", ctypes.c_int64), ("threads", ctypes.c_int32),
                ("vectors_per_thread", ctypes.c_int32)]


MAP_NAMES = {0: "linear", 1: "xcd_groups", 2: "xcd_pages", 3: "xcd_lists", 4: "xcd_shards"}


class NapTopology(ctypes.Structure):
    """Mirror of nuna_nap_topology_t."""
    _fields_ = [("num_domains", ctypes.c_int32), ("cus_per_domain", ctypes.c_int32),
                ("num_stacks", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("cu_budget", ctypes.c_int64), ("stack_budget", ctypes.c_int64),
                ("stack_pref", (ctypes.c_int32 * NAP_MAX_STACKS) * NAP_MAX_DOMAINS)]

# Every function the header declares, with its ctypes signature.
SIGNATURES = {
    "nuna_init": ([], ctypes.c_int),
    "nuna_get_device_info": ([ctypes.POINTER(DeviceInfo)], ctypes.c_int),
    "nuna_last_launch": ([ctypes.POINTER(LaunchInfo)], ctypes.c_int),
    "nuna_check_dispatch_map": ([_i32p, ctypes.c_int64, ctypes.c_int32], ctypes.c_int),
    "nuna_last_error_string": ([], ctypes.c_char_p),
    "nuna_version": ([], ctypes.c_int),
    "nuna_set_max_workgroups": ([ctypes.c_int], ctypes.c_int),
    "nuna_set_tunable": ([ctypes.c_char_p, ctypes.c_int64], ctypes.c_int),
    "nuna_get_tunable": ([ctypes.c_char_p, _i64p], ctypes.c_int),
    "nuna_allreduce": ([_vpp, _vpp, ctypes.c_int, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp],
                       ctypes.c_int),
    "nuna_reduce_scatter": ([_vpp, _vpp, ctypes.c_int, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, _vp],
                            ctypes.c_int),
    "nuna_all_gather": ([_vpp, _vpp, ctypes.c_int, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, _vp], ctypes.c_int),
    "nuna_a2a_layout_create": ([ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp,
                                ctypes.POINTER(_vp)], ctypes.c_int),
    "nuna_a2a_layout_upload": ([_vp], ctypes.c_int),
    "nuna_a2a_layout_recv_rows": ([_vp, _i64p], ctypes.c_int),
    "nuna_a2a_layout_recv_map": ([_vp, ctypes.c_int, _i32p, _i32p], ctypes.c_int),
    "nuna_a2a_layout_destroy": ([_vp], None),
    "nuna_all_to_all": ([_vpp, _vpp, _vp, ctypes.c_size_t, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, _vp],
                        ctypes.c_int),
    "nuna_all_to_all_routed": ([_vpp, _vpp, _vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                ctypes.c_size_t, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, _vp, _vp], ctypes.c_int),
    "nuna_all_to_all_combine": ([_vpp, _vpp, _vp, _vp, ctypes.c_size_t, ctypes.c_size_t, ctypes.c_int,
                                 ctypes.c_int, _vp], ctypes.c_int),
    "nuna_placement_items": ([ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, _i64p,
                              ctypes.c_int64, _i64p], ctypes.c_int),
    "nuna_placement_grid": ([ctypes.c_int, ctypes.c_int64, ctypes.c_int64, _i64p], ctypes.c_int),
    "nuna_placement_direct": ([ctypes.c_int, ctypes.c_int64, ctypes.c_int64, _i64p, ctypes.c_int64, _i64p],
                              ctypes.c_int),
    "nuna_probe_xcc": ([ctypes.c_int, _vp, _vp, _vp], ctypes.c_int),
    "nuna_copy": ([_vp, _vp, ctypes.c_size_t, _vp], ctypes.c_int),
    "nuna_ref_stream": ([ctypes.c_int, _vpp, _vpp, ctypes.c_int, ctypes.c_size_t, _vp], ctypes.c_int),
    "nuna_nap_topology_mi355x": ([ctypes.POINTER(NapTopology)], ctypes.c_int),
    "nuna_nap_plan": ([ctypes.POINTER(NapTopology), ctypes.c_int, ctypes.c_int64, _i64p, _i64p, _i64p, _i64p,
                       _i64p, _i32p, _i32p, _i32p, _i64p], ctypes.c_int),
    "nuna_probe_load_latency_cus": ([_vp, ctypes.c_size_t, ctypes.c_size_t, ctypes.c_int, _vp, _vp, _vp, _vp],
                                    ctypes.c_int),
    "nuna_probe_load_latency": ([_vp, ctypes.c_size_t, ctypes.c_size_t, ctypes.c_size_t, ctypes.c_int, _vp, _vp],
                                ctypes.c_int),
}

_lib = None


class NunaError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def lib():
    """Load libnuna.so once.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def last_error():
    return lib().nuna_last_error_string().decode()


def _check(st):
    if st != OK:
        raise NunaError(st, last_error())


def _ptr_array(ptrs):
    return (ctypes.c_void_p * max(len(ptrs), 1))(*[int(p) if p is not None else None for p in ptrs])


# ------------------------------------------------------------------ raw ABI (integer pointers)

def allreduce_raw(in_ptrs, out_ptrs, P, count, dtype, algo=ALGO_AUTO, place=XCD, stream=0):
    a = _ptr_array(in_ptrs) if in_ptrs is not None else None
    b = _ptr_array(out_ptrs) if out_ptrs is not None else None
    return lib().nuna_allreduce(a, b, P, count, dtype, algo, place, stream)


def reduce_scatter_raw(in_ptrs, out_ptrs, P, recvcount, dtype, place=XCD, stream=0):
    a = _ptr_array(in_ptrs) if in_ptrs is not None else None
    b = _ptr_array(out_ptrs) if out_ptrs is not None else None
    return lib().nuna_reduce_scatter(a, b, P, recvcount, dtype, place, stream)


def all_gather_raw(in_ptrs, out_ptrs, P, sendcount, dtype, place=XCD, stream=0):
    a = _ptr_array(in_ptrs) if in_ptrs is not None else None
    b = _ptr_array(out_ptrs) if out_ptrs is not None else None
    return lib().nuna_all_gather(a, b, P, sendcount, dtype, place, stream)


def all_to_all_raw(send_ptrs, recv_ptrs, layout_handle, row_elems, recv_capacity_rows, dtype, place=XCD, stream=0):
    a = _ptr_array(send_ptrs) if send_ptrs is not None else None
    b = _ptr_array(recv_ptrs) if recv_ptrs is not None else None
    return lib().nuna_all_to_all(a, b, layout_handle, row_elems, recv_capacity_rows, dtype, place, stream)


def all_to_all_combine_raw(y_ptrs, out_ptrs, layout_handle, row_elems, y_capacity_rows, dtype, place=XCD, stream=0,
                           weights_ptr=None):
    a = _ptr_array(y_ptrs) if y_ptrs is not None else None
    b = _ptr_array(out_ptrs) if out_ptrs is not None else None
    return lib().nuna_all_to_all_combine(a, b, layout_handle, weights_ptr, row_elems, y_capacity_rows, dtype, place,
                                         stream)


def placement_items(place, b, G, groups, group_size):
    """Work items workgroup b of G runs, in order (host mirror of the kernels' map)."""
    import numpy as np
    cnt = ctypes.c_int64()
    lib().nuna_placement_items(PLACEMENTS[place], b, G, groups, group_size, None, 0, ctypes.byref(cnt))
    n = cnt.value
    buf = np.zeros(max(n, 1), dtype=np.int64)
    _check(lib().nuna_placement_items(PLACEMENTS[place], b, G, groups, group_size, buf.ctypes.data_as(_i64p), n,
                                      ctypes.byref(cnt)))
    return buf[:n].tolist()


def placement_grid(place, groups, group_size):
    """Workgroups a launch of this placement uses (before the cap)."""
    g = ctypes.c_int64()
    _check(lib().nuna_placement_grid(PLACEMENTS[place], groups, group_size, ctypes.byref(g)))
    return g.value


def placement_direct(place, items, chunk_bytes):
    """Item each workgroup of a one-item-per-workgroup launch runs (-1: padding), host mirror."""
    import numpy as np
    g = ctypes.c_int64()
    lib().nuna_placement_direct(PLACEMENTS[place], items, chunk_bytes, None, 0, ctypes.byref(g))
    buf = np.zeros(max(g.value, 1), dtype=np.int64)
    _check(lib().nuna_placement_direct(PLACEMENTS[place], items, chunk_bytes, buf.ctypes.data_as(_i64p), g.value,
                                       ctypes.byref(g)))
    return buf[:g.value]


def nap_topology_mi355x(cu_budget=None, stack_budget=None):
    """The library's MI355X topology for the placement planner, budgets optionally replaced."""
    t = NapTopology()
    _check(lib().nuna_nap_topology_mi355x(ctypes.byref(t)))
    if cu_budget is not None:
        t.cu_budget = int(cu_budget)
    if stack_budget is not None:
        t.stack_budget = int(stack_budget)
    return t


def nap_plan(tb_chunks, tb_bytes, nar_max, topo=None, entry_pages=None):
    """Algorithm 1 in the library: tb_chunks is a list of chunk-id lists (one per threadblock),
    tb_bytes the charge of each.  Returns numpy arrays tb_group, tb_domain, tb_cu, entry_stack
    (aligned with the flattened chunk lists) and the group count."""
    import numpy as np
    topo = nap_topology_mi355x() if topo is None else topo
    n = len(tb_chunks)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(c) for c in tb_chunks])
    ids = np.array([c for cs in tb_chunks for c in cs], dtype=np.int64)
    cs = np.ascontiguousarray(tb_bytes, dtype=np.int64)
    pages = None if entry_pages is None else np.ascontiguousarray(entry_pages, dtype=np.int64)
    g = np.zeros(n, dtype=np.int64)
    d = np.zeros(n, dtype=np.int32)
    cu = np.zeros(n, dtype=np.int32)
    st = np.zeros(max(1, ids.size), dtype=np.int32)
    ng = ctypes.c_int64()
    ptr = lambda a, t: a.ctypes.data_as(t) if a is not None and a.size else None  # noqa: E731
    _check(lib().nuna_nap_plan(ctypes.byref(topo), int(nar_max), n, ptr(off, _i64p), ptr(ids, _i64p),
                               ptr(cs, _i64p), ptr(pages, _i64p), ptr(g, _i64p), ptr(d, _i32p), ptr(cu, _i32p),
                               ptr(st, _i32p), ctypes.byref(ng)))
    return {"tb_group": g, "tb_domain": d, "tb_cu": cu, "entry_stack": st[:ids.size], "num_groups": ng.value}


def set_tunable(name, value):
    """Set a launch-shape tunable (NUNA_* name) for later calls; never changes results."""
    _check(lib().nuna_set_tunable(name.encode(), int(value)))


def get_tunable(name):
    v = ctypes.c_int64()
    _check(lib().nuna_get_tunable(name.encode(), ctypes.byref(v)))
    return v.value


class tunables:
    """Context manager: set tunables on entry, restore the previous values on exit."""

    def __init__(self, **values):
        self.values = values
        self.saved = {}

    def __enter__(self):
        for k, v in self.values.items():
            self.saved[k] = get_tunable(k)
            set_tunable(k, v)
        return self

    def __exit__(self, *exc):
        for k, v in self.saved.items():
            set_tunable(k, v)
        return False


def init():
    """Probe the current device (architecture, dispatch map); XCD placement needs it."""
    _check(lib().nuna_init())


def device_info():
    """What nuna_init found on the current device: dict of device, cu_count, xcd_count, map_verified."""
    info = DeviceInfo()
    _check(lib().nuna_get_device_info(ctypes.byref(info)))
    return {k: int(getattr(info, k)) for k, _ in DeviceInfo._fields_}


def last_launch():
    """Kernels and map of the calling thread's last collective call (dict)."""
    info = LaunchInfo()
    _check(lib().nuna_last_launch(ctypes.byref(info)))
    d = {k: getattr(info, k) for k, _ in LaunchInfo._fields_}
    d["kernels"] = info.kernels.decode()
    d["map"] = MAP_NAMES.get(int(info.map), int(info.map))
    return d


def check_dispatch_map_raw(xcc, cu_count):
    """Status of the library's host-side dispatch-map check on an int32 array of per-workgroup XCC ids."""
    import numpy as np
    a = np.ascontiguousarray(xcc, dtype=np.int32)
    return lib().nuna_check_dispatch_map(a.ctypes.data_as(_i32p) if a.size else None, int(a.size), int(cu_count))


def set_max_workgroups(n):
    """Cap workgroups per launch (0 = default); launch shape only, never results."""
    _check(lib().nuna_set_max_workgroups(int(n)))


# ------------------------------------------------------------------ tensor API

def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _check_ranks(ts, name):
    if not ts:
        raise ValueError(f"{name}: need at least one rank buffer")
    d, n = ts[0].dtype, ts[0].numel()
    for t in ts:
        if not t.is_cuda or not t.is_contiguous() or t.dtype != d or t.numel() != n:
            raise ValueError(f"{name}: rank buffers must be contiguous CUDA tensors of one dtype and size")
    return d, n


def _check_outs(ins, outs, n_out):
    """One output per input rank, each of the input dtype and n_out elements: checked before any
    pointer reaches the library, which sizes every output from the input dtype."""
    if len(outs) != len(ins):
        raise ValueError(f"need one output per rank: {len(outs)} outputs for {len(ins)} inputs")
    for o in outs:
        if o.dtype != ins[0].dtype:
            raise ValueError(f"output dtype {o.dtype} differs from input dtype {ins[0].dtype}")
        if o.numel() != n_out:
            raise ValueError(f"each output holds {n_out} elements, got {o.numel()}")


def allreduce(ins, outs=None, algo="auto", placement="xcd", stream=None):
    """out[d] = sum over ranks r (ascending, fp32 accumulation) of ins[r], for every d."""
    _, n = _check_ranks(ins, "ins")
    if outs is None:
        outs = [_torch().empty_like(ins[0]) for _ in ins]
    _check_outs(ins, outs, n)
    _check_ranks(outs, "outs")
    _check(allreduce_raw([t.data_ptr() for t in ins], [t.data_ptr() for t in outs], len(ins), n,
                         _dtype_code(ins[0]), ALGOS[algo], PLACEMENTS[placement], _stream(stream)))
    return outs


class Prepared:
    """A collective call whose buffers were checked and whose arguments were marshalled once.
    Calling it launches the collective again, on `stream` (a torch stream, a raw stream handle, or
    None for torch's current stream), with no per-call Python checks.  The tensors it was built
    from must stay alive and keep their storage; they are held by this object."""

    def __init__(self, fn, args, keep):
        self._fn = fn
        self._args = args
        self._keep = keep

    def __call__(self, stream=None):
        if stream is None:
            h = _torch().cuda.current_stream().cuda_stream
        elif isinstance(stream, int):
            h = stream
        else:
            h = stream.cuda_stream
        _check(self._fn(*self._args, h))


def prepare_allreduce(ins, outs, algo="auto", placement="xcd"):
    """allreduce(ins, outs, algo, placement) as a Prepared call."""
    _, n = _check_ranks(ins, "ins")
    _check_outs(ins, outs, n)
    _check_ranks(outs, "outs")
    a = _ptr_array([t.data_ptr() for t in ins])
    b = _ptr_array([t.data_ptr() for t in outs])
    args = (a, b, len(ins), n, _dtype_code(ins[0]), ALGOS[algo], PLACEMENTS[placement])
    return Prepared(lib().nuna_allreduce, args, (list(ins), list(outs)))


def reduce_scatter(ins, outs=None, placement="xcd", stream=None):
    """outs[r][j] = sum over q ascending of ins[q][r*m + j], m = numel / P."""
    _, n = _check_ranks(ins, "ins")
    P = len(ins)
    if n % P:
        raise ValueError("reduce-scatter input size must be a multiple of P")
    m = n // P
    if outs is None:
        outs = [_torch().empty(m, dtype=ins[0].dtype, device=ins[0].device) for _ in ins]
    _check_outs(ins, outs, m)
    _check_ranks(outs, "outs")
    _check(reduce_scatter_raw([t.data_ptr() for t in ins], [t.data_ptr() for t in outs], P, m, _dtype_code(ins[0]),
                              PLACEMENTS[placement], _stream(stream)))
    return outs


def all_gather(ins, outs=None, placement="xcd", stream=None):
    """outs[d][r*m + j] = ins[r][j] for every d."""
    _, m = _check_ranks(ins, "ins")
    P = len(ins)
    if outs is None:
        outs = [_torch().empty(P * m, dtype=ins[0].dtype, device=ins[0].device) for _ in ins]
    _check_outs(ins, outs, P * m)
    _check_ranks(outs, "outs")
    _check(all_gather_raw([t.data_ptr() for t in ins], [t.data_ptr() for t in outs], P, m, _dtype_code(ins[0]),
                          PLACEMENTS[placement], _stream(stream)))
    return outs


class A2ALayout:
    """Routing plan of one MoE dispatch (host planning in the library)."""

    def __init__(self, topk_idx, num_experts):
        import numpy as np
        topk = np.ascontiguousarray(topk_idx, dtype=np.int32)
        if topk.ndim != 3:
            raise ValueError("topk_idx must be [P, tokens_per_rank, topk]")
        self.P, self.T, self.k = (int(x) for x in topk.shape)
        self.num_experts = int(num_experts)
        self._topk = topk
        h = ctypes.c_void_p()
        _check(lib().nuna_a2a_layout_create(self.P, self.T, self.k, self.num_experts,
                                            topk.ctypes.data if topk.size else None, ctypes.byref(h)))
        self.handle = h

    def upload(self):
        _check(lib().nuna_a2a_layout_upload(self.handle))
        return self

    def recv_rows(self):
        import numpy as np
        rows = np.zeros(self.P, dtype=np.int64)
        _check(lib().nuna_a2a_layout_recv_rows(self.handle, rows.ctypes.data_as(_i64p)))
        return rows

    def recv_map(self, d):
        import numpy as np
        n = int(self.recv_rows()[d])
        sr = np.zeros(max(n, 1), dtype=np.int32)
        st = np.zeros(max(n, 1), dtype=np.int32)
        _check(lib().nuna_a2a_layout_recv_map(self.handle, d, sr.ctypes.data_as(_i32p), st.ctypes.data_as(_i32p)))
        return sr[:n], st[:n]

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            lib().nuna_a2a_layout_destroy(self.handle)
        self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def all_to_all(send, recv, layout, placement="xcd", stream=None):
    """recv[d][j] = send[s][t] for the j-th row (s, t) routed to d by the layout."""
    P = layout.P
    if len(send) != P or len(recv) != P:
        raise ValueError("one send and one recv buffer per rank")
    for t in send:
        if not t.is_cuda or not t.is_contiguous() or t.dim() != 2 or t.shape != send[0].shape:
            raise ValueError("send buffers must be contiguous CUDA tensors [T, row]")
    row = send[0].shape[1]
    cap = recv[0].shape[0]
    for t in recv:
        if not t.is_cuda or not t.is_contiguous() or t.dim() != 2 or t.shape[1] != row or t.dtype != send[0].dtype:
            raise ValueError("recv buffers must be contiguous CUDA tensors [capacity, row] of the send dtype")
        cap = min(cap, t.shape[0])
    _check(all_to_all_raw([t.data_ptr() for t in send], [t.data_ptr() for t in recv], layout.handle, row, cap,
                          _dtype_code(send[0]), PLACEMENTS[placement], _stream(stream)))
    return recv


def all_to_all_routed_raw(send_ptrs, recv_ptrs, topk_ptr, P, T, k, E, row_elems, recv_capacity_rows, dtype,
                          rows_ptr, place=XCD, stream=0):
    a = _ptr_array(send_ptrs) if send_ptrs is not None else None
    b = _ptr_array(recv_ptrs) if recv_ptrs is not None else None
    return lib().nuna_all_to_all_routed(a, b, topk_ptr, P, T, k, E, row_elems, recv_capacity_rows, dtype, place,
                                        rows_ptr, stream)


def all_to_all_routed(send, recv, topk_idx, num_experts, rows_per_rank, placement="xcd", stream=None):
    """Dispatch with the routing on the device and no allocation: topk_idx an int32 CUDA tensor
    [P, T, k]; rows_per_rank an int64 CUDA tensor of P + 1 that receives the rows each rank gets
    (and, last, the count of out-of-range experts)."""
    torch = _torch()
    P = len(send)
    if len(recv) != P or topk_idx.dim() != 3 or topk_idx.shape[0] != P or topk_idx.dtype != torch.int32:
        raise ValueError("one send and one recv buffer per rank; topk_idx int32 [P, T, k]")
    if not topk_idx.is_cuda or not topk_idx.is_contiguous():
        raise ValueError("topk_idx must be a contiguous CUDA tensor")
    if (not rows_per_rank.is_cuda or rows_per_rank.dtype != torch.int64 or rows_per_rank.numel() != P + 1
            or not rows_per_rank.is_contiguous()):
        raise ValueError("rows_per_rank must be a contiguous int64 CUDA tensor of P + 1")
    T, k = int(topk_idx.shape[1]), int(topk_idx.shape[2])
    for t in send:
        if not t.is_cuda or not t.is_contiguous() or t.dim() != 2 or t.shape != (T, send[0].shape[1]):
            raise ValueError("send buffers must be contiguous CUDA tensors [T, row]")
    row = send[0].shape[1]
    cap = recv[0].shape[0]
    for t in recv:
        if not t.is_cuda or not t.is_contiguous() or t.dim() != 2 or t.shape[1] != row or t.dtype != send[0].dtype:
            raise ValueError("recv buffers must be contiguous CUDA tensors [capacity, row] of the send dtype")
        cap = min(cap, t.shape[0])
    _check(all_to_all_routed_raw([t.data_ptr() for t in send], [t.data_ptr() for t in recv], topk_idx.data_ptr(),
                                 P, T, k, int(num_experts), row, cap, _dtype_code(send[0]), rows_per_rank.data_ptr(),
                                 PLACEMENTS[placement], _stream(stream)))
    return recv


def all_to_all_combine(y, out, layout, placement="xcd", stream=None, weights=None):
    """out[s][t] = sum over the ranks d that token (s, t) was sent to (ascending) of its result row in y[d],
    each first scaled by weights[s, t, d] when weights (float32 CUDA tensor [P, T, P]) is given."""
    P = layout.P
    wp = None
    if weights is not None:
        if (not weights.is_cuda or weights.dtype != _torch().float32 or not weights.is_contiguous()
                or tuple(weights.shape) != (P, layout.T, P)):
            raise ValueError("weights must be a contiguous float32 CUDA tensor [P, T, P]")
        wp = weights.data_ptr()
    if len(y) != P or len(out) != P:
        raise ValueError("one result and one output buffer per rank")
    for t in out:
        if not t.is_cuda or not t.is_contiguous() or t.dim() != 2 or t.shape != out[0].shape:
            raise ValueError("output buffers must be contiguous CUDA tensors [T, row]")
    row = out[0].shape[1]
    cap = y[0].shape[0]
    for t in y:
        if not t.is_cuda or not t.is_contiguous() or t.dim() != 2 or t.shape[1] != row or t.dtype != out[0].dtype:
            raise ValueError("result buffers must be contiguous CUDA tensors [capacity, row] of the output dtype")
        cap = min(cap, t.shape[0])
    _check(all_to_all_combine_raw([t.data_ptr() for t in y], [t.data_ptr() for t in out], layout.handle, row, cap,
                                  _dtype_code(out[0]), PLACEMENTS[placement], _stream(stream), wp))
    return out


def probe_xcc(G, stream=None):
    """Run the dispatch probe: per workgroup, the XCC id and raw HW_ID it ran on."""
    torch = _torch()
    xcc = torch.full((G,), -1, dtype=torch.int32, device="cuda")
    hw = torch.full((G,), -1, dtype=torch.int32, device="cuda")
    _check(lib().nuna_probe_xcc(G, xcc.data_ptr(), hw.data_ptr(), _stream(stream)))
    return xcc, hw


def _check_flat(ts, name):
    """Each tensor is a contiguous CUDA tensor, so that its data pointer and numel() * element_size() bytes
    span exactly its own storage (an expanded or strided view would span more or other memory)."""
    for t in ts:
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name}: buffers must be contiguous CUDA tensors")


def copy(dst, src, stream=None):
    _check_flat((dst, src), "copy")
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < nbytes:
        raise ValueError("dst too small")
    _check(lib().nuna_copy(dst.data_ptr(), src.data_ptr(), nbytes, _stream(stream)))
    return dst


REF_KINDS = {"read": 0, "write": 1, "copy": 2}


def ref_read_checksum_bytes(n, nbytes):
    """Bytes a reference read of n buffers of nbytes writes to dst[0]: one 16-byte checksum per item of
    max(1, 8 // n) blocks of 4 KiB."""
    item = (1 if n >= 8 else 8 // n) * 4096
    return (nbytes + item - 1) // item * 16


def ref_stream_raw(kind, src_ptrs, dst_ptrs, n, nbytes, stream=0):
    """nuna_ref_stream on raw device addresses (lists of ints or None) and a raw stream handle;
    returns the status code."""
    src = _ptr_array(src_ptrs) if src_ptrs is not None else None
    dst = _ptr_array(dst_ptrs) if dst_ptrs is not None else None
    return lib().nuna_ref_stream(REF_KINDS[kind], src, dst, n, nbytes, stream)


def ref_stream(kind, srcs, dsts, stream=None):
    """Reference stream over CUDA tensors: "read" (srcs; dsts[0] receives ref_read_checksum_bytes of
    checksums), "write" (dsts), or "copy" (dsts[r] = srcs[r]).  Every buffer holds the same number of
    bytes."""
    if kind not in REF_KINDS:
        raise ValueError(f"reference stream kind {kind!r} is not one of {sorted(REF_KINDS)}")
    bufs = dsts if kind == "write" else srcs
    if not bufs or not dsts:
        raise ValueError("reference stream needs its buffers and at least one destination")
    _check_flat(list(bufs) + list(dsts), "ref_stream")
    nbytes = bufs[0].numel() * bufs[0].element_size()
    if any(b.numel() * b.element_size() != nbytes for b in bufs):
        raise ValueError("reference stream buffers differ in size")
    if kind == "read" and dsts[0].numel() * dsts[0].element_size() < ref_read_checksum_bytes(len(srcs), nbytes):
        raise ValueError("checksum buffer too small")
    if kind == "copy" and (len(dsts) != len(srcs) or any(d.numel() * d.element_size() < nbytes for d in dsts)):
        raise ValueError("copy destinations must match the sources")
    n = len(bufs)
    _check(ref_stream_raw(kind, None if kind == "write" else [s.data_ptr() for s in srcs],
                          [d.data_ptr() for d in dsts], n, nbytes, _stream(stream)))
    return dsts


def probe_load_latency(buf, stride, line_offset, xcd, stream=None):
    """Cold-load latency (shader cycles) of each stride-sized block of `buf` (a CUDA tensor) seen from
    XCD `xcd`.  The caller evicts the caches first.  Returns an int64 CPU tensor."""
    torch = _torch()
    _check_flat((buf,), "probe")
    nbytes = buf.numel() * buf.element_size()
    cyc = torch.zeros(nbytes // stride, dtype=torch.int32, device=buf.device)
    _check(lib().nuna_probe_load_latency(buf.data_ptr(), nbytes, stride, line_offset, xcd, cyc.data_ptr(),
                                         _stream(stream)))
    torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
    return cyc.cpu().to(torch.int64)


def memory_affinity(buf, stride=8192, line_offset=256, xcds=(0, 4), evict_bytes=1 << 30):
    """Near XCD group of each block of `buf`: probe it cold from one XCD of each group and return
    (latencies [len(xcds), nblocks] int64, near index per block).  Eviction between passes streams
    `evict_bytes` through a scratch tensor (plumbing on the host side of the call)."""
    torch = _torch()
    ev = torch.empty(evict_bytes // 4, dtype=torch.int32, device=buf.device)
    lats = []
    for j, x in enumerate(xcds):
        ev.fill_(j)
        torch.cuda.synchronize()
        lats.append(probe_load_latency(buf, stride, line_offset, x))
    del ev
    lat = torch.stack(lats)
    return lat, lat.argmin(dim=0)


def probe_load_latency_cus(buf, xcd, stride=8192, stream=None):
    """Cold-load latency (shader cycles) of every stride-sized block of `buf` from each compute unit of
    XCD `xcd` it reaches.  Returns (latencies int64 [cus, nblocks] on the CPU, HW_ID CU keys [cus],
    compute units seen).  The caller evicts the caches first."""
    torch = _torch()
    _check_flat((buf,), "probe")
    nbytes = buf.numel() * buf.element_size()
    nb = nbytes // stride
    work = torch.zeros(257, dtype=torch.int32, device=buf.device)
    cyc = torch.zeros((32, nb), dtype=torch.int32, device=buf.device)
    cu = torch.full((32,), -1, dtype=torch.int32, device=buf.device)
    _check(lib().nuna_probe_load_latency_cus(buf.data_ptr(), nbytes, stride, xcd, work.data_ptr(), cyc.data_ptr(),
                                             cu.data_ptr(), _stream(stream)))
    torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
    seen = int(work[256].item())
    n = min(seen, 32)
    return cyc[:n].cpu().to(torch.int64), cu[:n].cpu().to(torch.int64), seen


def cu_latency_map(buf, stride=8192, xcds=range(8), evict_bytes=1 << 30):
    """Per-XCD, per-compute-unit cold-load latencies over every block of `buf`: dict xcd ->
    (latencies [cus, nblocks], CU keys, compute units seen).  Caches are evicted before each XCD's
    pass by streaming `evict_bytes` through a scratch tensor (plumbing on the host side)."""
    torch = _torch()
    ev = torch.empty(evict_bytes // 4, dtype=torch.int32, device=buf.device)
    out = {}
    for j, x in enumerate(xcds):
        ev.fill_(j)
        torch.cuda.synchronize()
        out[x] = probe_load_latency_cus(buf, x, stride)
    del ev
    return out
