"""MI355X-native DualGCN aggregation: Python binding of ``libdualgcn.so``.

Argument marshalling only -- every step of the path runs in the library's HIP
kernels.  torch provides device memory and the current stream.  The library is
built by ``python paper_2609_01983_amd/build.py`` (or ``__graft_entry__.build()``); if it
is missing, importing this package raises ImportError: there is no fallback.

    plan = Plan(rowptr, col, val, seed=0, walks_per_node=16, walk_len=5)
    Y = spmm(plan, X)                           # Y = A X
    T = update(X, W)                            # T = X W, bf16 matrix cores
    H = gcn_layer(plan, X, W, relu=True)        # H = relu(A (X W)), X W in bf16 MFMA
"""
import ctypes
import os

import torch  # must load before the library: it provides the process's HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdualgcn.so")

OK, ERR_INVALID_ARG, ERR_BAD_CSR, ERR_UNSUPPORTED, ERR_OOM, ERR_HIP, ERR_NO_DEVICE = \
    0, -1, -2, -3, -4, -5, -6
FORCE_AUTO, FORCE_SPARSE, FORCE_DENSE = 0, 1, 2
RELU, OUT_BF16, IN_BF16, GRAD_BF16 = 1, 2, 4, 8
LOSS_SLOTS = 1025                # float64 entries of the loss buffer of softmax_xent
ALPHA_ADAPTIVE = 0xFFFFFFFF      # alpha = (ALPHA_ADAPTIVE, q): adaptive weight in steps of 1/q
ALPHA_BALANCED = 0xFFFFFFFE      # alpha = (ALPHA_BALANCED, q): weight balancing the spreads of N and D

_FORCE = {"auto": FORCE_AUTO, "sparse": FORCE_SPARSE, "dense": FORCE_DENSE,
          FORCE_AUTO: FORCE_AUTO, FORCE_SPARSE: FORCE_SPARSE, FORCE_DENSE: FORCE_DENSE}


class DualGCNError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {status_str(status)} ({status})"
                         + (f", hip error {_lib.dualgcn_last_hip_error()}" if status == ERR_HIP else ""))


class Csr(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("nnz", ctypes.c_int64), ("rowptr", ctypes.c_void_p),
                ("col", ctypes.c_void_p), ("val", ctypes.c_void_p)]


class Thresholds(ctypes.Structure):
    _fields_ = [("alpha_num", ctypes.c_uint32), ("alpha_den", ctypes.c_uint32),
                ("beta_num", ctypes.c_uint32), ("beta_den", ctypes.c_uint32),
                ("force_mode", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("nnz", ctypes.c_int64), ("n_sparse", ctypes.c_int32),
                ("n_dense", ctypes.c_int32), ("kstar", ctypes.c_uint64),
                ("s1_hi", ctypes.c_uint64), ("s1_lo", ctypes.c_uint64),
                ("s2_hi", ctypes.c_uint64), ("s2_lo", ctypes.c_uint64), ("kmax", ctypes.c_uint64),
                ("alpha_num", ctypes.c_uint32), ("alpha_den", ctypes.c_uint32),
                ("beta_num", ctypes.c_uint32), ("beta_den", ctypes.c_uint32),
                ("force_mode", ctypes.c_int32), ("seed", ctypes.c_uint64),
                ("walks_per_node", ctypes.c_uint32), ("walk_len", ctypes.c_uint32),
                ("max_degree", ctypes.c_int32), ("dense_chunk", ctypes.c_int32),
                ("n_split_rows", ctypes.c_int32), ("n_split_parts", ctypes.c_int32),
                ("n_tasks", ctypes.c_int32), ("n_long_rows", ctypes.c_int32),
                ("cold_marked", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2609_01983_amd/build.py`")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, U32, U64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64, \
        ctypes.c_size_t
    sig = {
        "dualgcn_status_str": ([ctypes.c_int], ctypes.c_char_p),
        "dualgcn_last_hip_error": ([], ctypes.c_int),
        "dualgcn_partition": ([ctypes.POINTER(Csr), U64, U32, U32, ctypes.POINTER(Thresholds), P,
                               ctypes.POINTER(P)], ctypes.c_int),
        "dualgcn_plan_destroy": ([P], None),
        "dualgcn_spmm": ([P, P, P, I32, P], ctypes.c_int),
        "dualgcn_spmm_act": ([P, P, P, I32, U32, P], ctypes.c_int),
        "dualgcn_spmm_update": ([P, P, P, P, P, I32, I32, U32, P], ctypes.c_int),
        "dualgcn_spmm_update_route": ([P, I32, I32, P], ctypes.c_int),
        "dualgcn_update": ([P, P, P, I32, I32, I32, U32, P], ctypes.c_int),
        "dualgcn_gcn_layer_workspace": ([P, I32, I32, ctypes.POINTER(SZ)], ctypes.c_int),
        "dualgcn_gcn_layer": ([P, P, P, P, I32, I32, U32, P, SZ, P], ctypes.c_int),
        "dualgcn_plan_query": ([P, ctypes.POINTER(PlanInfo)], ctypes.c_int),
        "dualgcn_plan_export": ([P, P, P, P], ctypes.c_int),
        "dualgcn_arw_patterns": ([ctypes.POINTER(Csr), U64, U32, U32, P, P], ctypes.c_int),
        "dualgcn_plan_save": ([P, P, ctypes.POINTER(SZ)], ctypes.c_int),
        "dualgcn_plan_load": ([ctypes.POINTER(Csr), P, SZ, P, ctypes.POINTER(P)], ctypes.c_int),
        "dualgcn_aggregator_values": ([ctypes.POINTER(Csr), I32, ctypes.c_float, P, P], ctypes.c_int),
        "dualgcn_softmax_xent": ([P, P, I32, I32, ctypes.c_float, P, P, P], ctypes.c_int),
        "dualgcn_weight_grad_workspace": ([I32, I32, I32, ctypes.POINTER(SZ)], ctypes.c_int),
        "dualgcn_weight_grad": ([P, P, P, I32, I32, I32, U32, ctypes.c_float, P, P, SZ, P],
                                ctypes.c_int),
        "dualgcn_weight_grad_noalloc": ([P, P, P, I32, I32, I32, U32, ctypes.c_float, P, P],
                                        ctypes.c_int),
        "dualgcn_backward_data": ([P, P, P, P, I32, I32, I32, U32, P], ctypes.c_int),
        "dualgcn_bandwidth_probe": ([I32, P, P, SZ, P], ctypes.c_int),
        "dualgcn_bandwidth_probe_out_floats": ([], I32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    return L


_lib = _load()


def lib():
    return _lib


def status_str(status):
    return _lib.dualgcn_status_str(status).decode()


def _check(status, what):
    if status != OK:
        raise DualGCNError(status, what)


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, dtype, name):
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def make_csr(rowptr, col, val):
    _dev(rowptr, torch.int32, "rowptr")
    _dev(col, torch.int32, "col")
    _dev(val, torch.float32, "val")
    n = rowptr.numel() - 1
    return Csr(n, col.numel(), rowptr.data_ptr(), col.data_ptr() if col.numel() else None,
               val.data_ptr() if val.numel() else None)


class Plan:
    """The dual-metric partition of one CSR matrix (device arrays, borrowed)."""

    def __init__(self, rowptr, col, val, seed=0, walks_per_node=16, walk_len=5,
                 alpha=(1, 2), beta=(1, 2), force_mode="auto", stream=None):
        self._keep = (rowptr, col, val)        # the plan borrows these arrays
        self.csr = make_csr(rowptr, col, val)
        self.n = self.csr.n
        th = Thresholds(alpha[0], alpha[1], beta[0], beta[1], _FORCE[force_mode])
        out = ctypes.c_void_p()
        _check(_lib.dualgcn_partition(ctypes.byref(self.csr), seed, walks_per_node, walk_len,
                                      ctypes.byref(th), _stream(stream), ctypes.byref(out)),
               "dualgcn_partition")
        self._h = out

    @property
    def handle(self):
        if not self._h:
            raise ValueError("plan destroyed")
        return self._h

    def info(self):
        pi = PlanInfo()
        _check(_lib.dualgcn_plan_query(self.handle, ctypes.byref(pi)), "dualgcn_plan_query")
        d = {name: getattr(pi, name) for name, _ in PlanInfo._fields_}
        d["s1"] = (d.pop("s1_hi") << 64) | d.pop("s1_lo")
        d["s2"] = (d.pop("s2_hi") << 64) | d.pop("s2_lo")
        return d

    def export(self):
        """(perm int32[n], S uint32[n], K uint64[n]) as numpy arrays."""
        import numpy as np
        perm = np.empty(self.n, dtype=np.int32)
        S = np.empty(self.n, dtype=np.uint32)
        K = np.empty(self.n, dtype=np.uint64)
        _check(_lib.dualgcn_plan_export(self.handle, perm.ctypes.data, S.ctypes.data,
                                        K.ctypes.data), "dualgcn_plan_export")
        return perm, S, K

    def save(self):
        """The plan as bytes (parameters, checksum of the structure, density sums)."""
        nbytes = ctypes.c_size_t()
        _check(_lib.dualgcn_plan_save(self.handle, None, ctypes.byref(nbytes)), "dualgcn_plan_save")
        buf = ctypes.create_string_buffer(nbytes.value)
        _check(_lib.dualgcn_plan_save(self.handle, buf, ctypes.byref(nbytes)), "dualgcn_plan_save")
        return buf.raw[:nbytes.value]

    @classmethod
    def load(cls, rowptr, col, val, blob, stream=None):
        """Rebuilds a saved plan on the same structure (values may differ), without walks."""
        self = cls.__new__(cls)
        self._keep = (rowptr, col, val)
        self.csr = make_csr(rowptr, col, val)
        self.n = self.csr.n
        out = ctypes.c_void_p()
        buf = ctypes.create_string_buffer(bytes(blob), len(blob))
        _check(_lib.dualgcn_plan_load(ctypes.byref(self.csr), buf, len(blob), _stream(stream),
                                      ctypes.byref(out)), "dualgcn_plan_load")
        self._h = out
        return self

    def destroy(self):
        if getattr(self, "_h", None):
            _lib.dualgcn_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def spmm(plan, X, Y=None, relu=False, out_bf16=False, stream=None):
    """Y = A X (or relu(A X)) on the plan's matrix.  X: float32 [n, F] on the device.

    With out_bf16, Y is bfloat16: the nearest-even rounding of the float32 result."""
    _dev(X, torch.float32, "X")
    if X.dim() != 2 or X.shape[0] != plan.n:
        raise ValueError("X must be [n, F]")
    ydt = torch.bfloat16 if out_bf16 else torch.float32
    if Y is None:
        Y = torch.empty(X.shape, dtype=ydt, device=X.device)
    _dev(Y, ydt, "Y")
    if Y.shape != X.shape:
        raise ValueError("Y must have X's shape")
    if relu or out_bf16:
        flags = (RELU if relu else 0) | (OUT_BF16 if out_bf16 else 0)
        _check(_lib.dualgcn_spmm_act(plan.handle, X.data_ptr(), Y.data_ptr(), X.shape[1], flags,
                                     _stream(stream)), "dualgcn_spmm_act")
    else:
        _check(_lib.dualgcn_spmm(plan.handle, X.data_ptr(), Y.data_ptr(), X.shape[1],
                                 _stream(stream)), "dualgcn_spmm")
    return Y


def update(X, W, T=None, stream=None):
    """T = X W on the bf16 matrix cores (float32 accumulation).  X: [n, F_in] float32 or
    bfloat16, W: [F_in, F_out] float32.

    Needs no plan: it may run on another stream while a partition is built."""
    if not isinstance(X, torch.Tensor) or X.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("X must be a float32 or bfloat16 tensor")
    _dev(X, X.dtype, "X")
    _dev(W, torch.float32, "W")
    F_in, F_out = W.shape
    if X.dim() != 2 or X.shape[1] != F_in:
        raise ValueError("X must be [n, F_in]")
    n = X.shape[0]
    if T is None:
        T = torch.empty((n, F_out), dtype=torch.float32, device=X.device)
    _dev(T, torch.float32, "T")
    if T.shape != (n, F_out):
        raise ValueError("T must be [n, F_out]")
    flags = IN_BF16 if X.dtype == torch.bfloat16 else 0
    _check(_lib.dualgcn_update(X.data_ptr(), W.data_ptr(), T.data_ptr(), n, F_in, F_out, flags,
                               _stream(stream)), "dualgcn_update")
    return T


def spmm_update_route(plan, F_in, F_out):
    """True when the fused kernel is the faster route of spmm_update on this plan and shape."""
    fused = ctypes.c_int32()
    _check(_lib.dualgcn_spmm_update_route(plan.handle, F_in, F_out, ctypes.byref(fused)),
           "dualgcn_spmm_update_route")
    return bool(fused.value)


def spmm_update(plan, X, W, T=None, relu=False, H=None, stream=None):
    """T = bf16(act(A X)) bf16(W) (float32 accumulation): the aggregation of one layer fused
    with the next layer's update.  X: float32 [n, F_in], W: float32 [F_in, F_out],
    T: float32 [n, F_out].  H: None (act(A X) is not kept), or a bfloat16 [n, F_in]
    tensor that receives bf16(act(A X)).  Where the library's two-call route is the faster
    one and no H is given, a temporary H is allocated for it (the same T either way)."""
    _dev(X, torch.float32, "X")
    _dev(W, torch.float32, "W")
    if X.dim() != 2 or X.shape[0] != plan.n:
        raise ValueError("X must be [n, F_in]")
    F_in, F_out = W.shape
    if X.shape[1] != F_in:
        raise ValueError("W must be [F_in, F_out]")
    if T is None:
        T = torch.empty((plan.n, F_out), dtype=torch.float32, device=X.device)
    _dev(T, torch.float32, "T")
    if T.shape != (plan.n, F_out):
        raise ValueError("T must be [n, F_out]")
    hp = None
    if H is not None:
        _dev(H, torch.bfloat16, "H")
        if H.shape != (plan.n, F_in):
            raise ValueError("H must be [n, F_in]")
        hp = H.data_ptr()
    elif not spmm_update_route(plan, F_in, F_out):
        hp = torch.empty((plan.n, F_in), dtype=torch.bfloat16, device=X.device).data_ptr()
    _check(_lib.dualgcn_spmm_update(plan.handle, X.data_ptr(), W.data_ptr(), T.data_ptr(), hp,
                                    F_in, F_out, RELU if relu else 0, _stream(stream)),
           "dualgcn_spmm_update")
    return T


def gcn_layer_workspace_bytes(plan, F_in, F_out):
    nbytes = ctypes.c_size_t()
    _check(_lib.dualgcn_gcn_layer_workspace(plan.handle, F_in, F_out, ctypes.byref(nbytes)),
           "dualgcn_gcn_layer_workspace")
    return nbytes.value


def gcn_layer(plan, X, W, relu=False, Y=None, workspace=None, out_bf16=False, stream=None):
    """Y = act(A (X W)) with X W on the bf16 matrix cores (float32 accumulation).

    X may be float32 or bfloat16; with out_bf16 Y is the bfloat16 rounding of the result."""
    if not isinstance(X, torch.Tensor) or X.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("X must be a float32 or bfloat16 tensor")
    _dev(X, X.dtype, "X")
    _dev(W, torch.float32, "W")
    F_in, F_out = W.shape
    if X.shape != (plan.n, F_in):
        raise ValueError("X must be [n, F_in]")
    ydt = torch.bfloat16 if out_bf16 else torch.float32
    if Y is None:
        Y = torch.empty((plan.n, F_out), dtype=ydt, device=X.device)
    _dev(Y, ydt, "Y")
    need = gcn_layer_workspace_bytes(plan, F_in, F_out)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=X.device)
    _dev(workspace, torch.uint8, "workspace")
    flags = (RELU if relu else 0) | (IN_BF16 if X.dtype == torch.bfloat16 else 0) | \
        (OUT_BF16 if out_bf16 else 0)
    _check(_lib.dualgcn_gcn_layer(plan.handle, X.data_ptr(), W.data_ptr(), Y.data_ptr(), F_in,
                                  F_out, flags, workspace.data_ptr(),
                                  workspace.numel(), _stream(stream)), "dualgcn_gcn_layer")
    return Y


# ------------------------------------------------------------------ aggregators

AGG_GCN, AGG_MEAN, AGG_SUM = 0, 1, 2
_AGG = {"gcn": AGG_GCN, "mean": AGG_MEAN, "sum": AGG_SUM,
        AGG_GCN: AGG_GCN, AGG_MEAN: AGG_MEAN, AGG_SUM: AGG_SUM}


def aggregator_values(rowptr, col, kind="gcn", eps=0.0, val=None, stream=None):
    """float32 values of an aggregation matrix on this structure: "gcn" 1/sqrt(d_r d_c),
    "mean" 1/d_r, "sum" 1 with 1 + eps on self-loops (GIN).  Validates the CSR (waits)."""
    if val is None:
        val = torch.empty(col.numel(), dtype=torch.float32, device=col.device)
    csr = make_csr(rowptr, col, val)
    _check(_lib.dualgcn_aggregator_values(ctypes.byref(csr), _AGG[kind], float(eps),
                                          val.data_ptr() if val.numel() else None,
                                          _stream(stream)), "dualgcn_aggregator_values")
    return val


# ------------------------------------------------------------------ training

def _float_or_bf16(t, name):
    if not isinstance(t, torch.Tensor) or t.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError(f"{name} must be a float32 or bfloat16 tensor")
    _dev(t, t.dtype, name)
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D")


def softmax_xent(Y, labels, scale=None, G=None, loss=None, stream=None):
    """Softmax cross-entropy over the rows whose label is in [0, C).

    Returns (G, loss): G = dloss/dY (float32 [n, C]) and a float64 device tensor of
    LOSS_SLOTS entries whose entry 0 is the loss.  scale defaults to 1 / (labeled rows),
    counted on the host from `labels` only when not given."""
    _dev(Y, torch.float32, "Y")
    _dev(labels, torch.int32, "labels")
    n, C = Y.shape
    if labels.shape != (n,):
        raise ValueError("labels must be [n]")
    if scale is None:
        scale = 1.0 / max(1, int(((labels >= 0) & (labels < C)).sum().item()))
    if G is None:
        G = torch.empty_like(Y)
    _dev(G, torch.float32, "G")
    if loss is None:
        loss = torch.empty(LOSS_SLOTS, dtype=torch.float64, device=Y.device)
    _dev(loss, torch.float64, "loss")
    if G.shape != Y.shape or loss.numel() < LOSS_SLOTS:
        raise ValueError("G must match Y and loss must hold LOSS_SLOTS entries")
    _check(_lib.dualgcn_softmax_xent(Y.data_ptr(), labels.data_ptr(), n, C, float(scale),
                                     G.data_ptr(), loss.data_ptr(), _stream(stream)),
           "dualgcn_softmax_xent")
    return G, loss


def weight_grad_workspace_bytes(n, F_in, F_out):
    nbytes = ctypes.c_size_t()
    _check(_lib.dualgcn_weight_grad_workspace(n, F_in, F_out, ctypes.byref(nbytes)),
           "dualgcn_weight_grad_workspace")
    return nbytes.value


def weight_grad(X, G, dW=None, lr=0.0, W=None, workspace=None, stream=None):
    """dW = X^T G on the bf16 matrix cores; with W, also the SGD step W -= lr dW.
    X: [n, F_in] and G: [n, F_out], each float32 or bfloat16."""
    _float_or_bf16(X, "X")
    _float_or_bf16(G, "G")
    n, F_in = X.shape
    if G.shape[0] != n:
        raise ValueError("X and G must have the same rows")
    F_out = G.shape[1]
    if dW is None:
        dW = torch.empty((F_in, F_out), dtype=torch.float32, device=X.device)
    _dev(dW, torch.float32, "dW")
    if W is not None:
        _dev(W, torch.float32, "W")
        if W.shape != (F_in, F_out):
            raise ValueError("W must be [F_in, F_out]")
    if dW.shape != (F_in, F_out):
        raise ValueError("dW must be [F_in, F_out]")
    need = weight_grad_workspace_bytes(n, F_in, F_out)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=X.device)
    flags = (IN_BF16 if X.dtype == torch.bfloat16 else 0) | \
            (GRAD_BF16 if G.dtype == torch.bfloat16 else 0)
    _check(_lib.dualgcn_weight_grad(X.data_ptr(), G.data_ptr(), dW.data_ptr(), n, F_in, F_out,
                                    flags, float(lr), W.data_ptr() if W is not None else None,
                                    workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                    _stream(stream)), "dualgcn_weight_grad")
    return dW


def weight_grad_noalloc(X, G, dW, lr=0.0, W=None, stream=None):
    """dualgcn_weight_grad_noalloc: weight_grad with the partial products in the library's
    static device array (no workspace, nothing allocated by the library).  dW [F_in, F_out]
    float32 is the caller's."""
    _float_or_bf16(X, "X")
    _float_or_bf16(G, "G")
    n, F_in = X.shape
    if G.shape[0] != n:
        raise ValueError("X and G must have the same rows")
    F_out = G.shape[1]
    _dev(dW, torch.float32, "dW")
    if dW.shape != (F_in, F_out):
        raise ValueError("dW must be [F_in, F_out]")
    if W is not None:
        _dev(W, torch.float32, "W")
        if W.shape != (F_in, F_out):
            raise ValueError("W must be [F_in, F_out]")
    flags = (IN_BF16 if X.dtype == torch.bfloat16 else 0) | \
            (GRAD_BF16 if G.dtype == torch.bfloat16 else 0)
    _check(_lib.dualgcn_weight_grad_noalloc(X.data_ptr(), G.data_ptr(), dW.data_ptr(), n, F_in,
                                            F_out, flags, float(lr),
                                            W.data_ptr() if W is not None else None,
                                            _stream(stream)), "dualgcn_weight_grad_noalloc")
    return dW


def backward_data(G, W, M=None, dX=None, stream=None):
    """dX = (G W^T) * [M > 0] on the bf16 matrix cores (no mask without M).
    G: [n, F_out] float32 or bfloat16, W: [F_in, F_out] float32, M: [n, F_in]."""
    _float_or_bf16(G, "G")
    _dev(W, torch.float32, "W")
    F_in, F_out = W.shape
    n = G.shape[0]
    if G.shape[1] != F_out:
        raise ValueError("G must be [n, F_out]")
    flags = GRAD_BF16 if G.dtype == torch.bfloat16 else 0
    if M is not None:
        _float_or_bf16(M, "M")
        if M.shape != (n, F_in):
            raise ValueError("M must be [n, F_in]")
        flags |= IN_BF16 if M.dtype == torch.bfloat16 else 0
    if dX is None:
        dX = torch.empty((n, F_in), dtype=torch.float32, device=G.device)
    _dev(dX, torch.float32, "dX")
    if dX.shape != (n, F_in):
        raise ValueError("dX must be [n, F_in]")
    _check(_lib.dualgcn_backward_data(G.data_ptr(), W.data_ptr(),
                                      M.data_ptr() if M is not None else None, dX.data_ptr(), n,
                                      F_in, F_out, flags, _stream(stream)), "dualgcn_backward_data")
    return dX


PROBE_COPY, PROBE_READ = 0, 1


def bandwidth_probe(kind, src, dst, stream=None):
    """dualgcn_bandwidth_probe: kind PROBE_COPY (dst = src) or PROBE_READ (src read once;
    dst receives per-workgroup sums, at least bandwidth_probe_out_floats() floats)."""
    nbytes = src.numel() * src.element_size()
    if kind == PROBE_COPY and dst.numel() * dst.element_size() < nbytes:
        raise ValueError("dst smaller than src")
    if kind == PROBE_READ and dst.numel() * dst.element_size() < 4 * _lib.dualgcn_bandwidth_probe_out_floats():
        raise ValueError("dst too small for the read probe's sums")
    _check(_lib.dualgcn_bandwidth_probe(kind, src.data_ptr(), dst.data_ptr(), nbytes, _stream(stream)),
           "dualgcn_bandwidth_probe")


def bandwidth_probe_out_floats():
    return int(_lib.dualgcn_bandwidth_probe_out_floats())


def arw_patterns(rowptr, col, val, seed, walks_per_node, walk_len, stream=None):
    """uint8 [n, k, d+1] anonymous walks (labels) of every node, on the device."""
    csr = make_csr(rowptr, col, val)
    out = torch.empty((csr.n, walks_per_node, walk_len + 1), dtype=torch.uint8,
                      device=rowptr.device)
    _check(_lib.dualgcn_arw_patterns(ctypes.byref(csr), seed, walks_per_node, walk_len,
                                     out.data_ptr(), _stream(stream)), "dualgcn_arw_patterns")
    return out


__all__ = ["Plan", "spmm", "spmm_update", "update", "gcn_layer", "gcn_layer_workspace_bytes", "arw_patterns",
           "DualGCNError", "lib", "status_str", "make_csr", "Csr", "Thresholds", "PlanInfo",
           "FORCE_AUTO", "FORCE_SPARSE", "FORCE_DENSE", "RELU", "OUT_BF16", "IN_BF16",
           "ALPHA_ADAPTIVE", "ALPHA_BALANCED", "GRAD_BF16", "LOSS_SLOTS", "softmax_xent", "weight_grad", "weight_grad_noalloc",
           "weight_grad_workspace_bytes", "backward_data", "aggregator_values", "AGG_GCN",
           "AGG_MEAN", "AGG_SUM", "bandwidth_probe", "bandwidth_probe_out_floats",
           "PROBE_COPY", "PROBE_READ"]
