"""Thin Python binding of libtabpack.so (argument marshalling only).

Every step of the packed training step, evaluation and selection runs in the
library's HIP kernels; PyTorch only provides device memory (the workspace and
the caller's tensors) and the current HIP stream.  Importing works without a
GPU; the library is loaded on first use and a missing library is an error
(there is no fallback path).
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtabpack.so")

PACK_OK = 0
TASKS = {"reg": 0, "bin": 1, "multi": 2}
PRECISIONS = {"bf16": 0, "fp32": 1}
PREDICT_MEMBERS, PREDICT_ENSEMBLE = 0, 1
STATUS_IDX_RANGE = 1
BIND_DATA_MAX_B = 2048  # PACK_BIND_DATA_MAX_B
OPTIMIZERS = {"adamw": 0, "muon": 1}

SYMBOLS = ["pack_last_error", "pack_init", "pack_destroy", "pack_get_hparams", "pack_workspace_size",
           "pack_bind", "pack_train_step", "pack_eval_members", "pack_select_workspace_size",
           "pack_select", "pack_member_param_count", "pack_get_params", "pack_set_params",
           "pack_get_grads", "pack_get_moments", "pack_debug_dropout_mask", "pack_debug_activation",
           "pack_profile_enable", "pack_profile_read", "pack_set_active", "pack_predict", "pack_status",
           "pack_stream_copy", "pack_select_static", "pack_bind_data"]


class MemberHP(ctypes.Structure):
    _fields_ = [("width", ctypes.c_int32), ("padded_width", ctypes.c_int32),
                ("drop_threshold", ctypes.c_uint32), ("depth", ctypes.c_int32),
                ("dropout", ctypes.c_double), ("lr", ctypes.c_double), ("wd", ctypes.c_double),
                ("scale", ctypes.c_double), ("muon_lr", ctypes.c_double), ("d_emb", ctypes.c_int32),
                ("reserved2", ctypes.c_int32), ("sigma", ctypes.c_double)]


class PackConfig(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("d_in", ctypes.c_int32), ("d_out", ctypes.c_int32),
                ("L", ctypes.c_int32), ("B", ctypes.c_int32), ("task", ctypes.c_int32),
                ("precision", ctypes.c_int32), ("width_lo", ctypes.c_int32),
                ("width_hi", ctypes.c_int32), ("quantum", ctypes.c_int32),
                ("decay_bias", ctypes.c_int32), ("keep_grads", ctypes.c_int32),
                ("dropout_lo", ctypes.c_double), ("dropout_hi", ctypes.c_double),
                ("lr_lo", ctypes.c_double), ("lr_hi", ctypes.c_double),
                ("wd_lo", ctypes.c_double), ("wd_hi", ctypes.c_double),
                ("beta1", ctypes.c_double), ("beta2", ctypes.c_double), ("eps", ctypes.c_double),
                ("seed", ctypes.c_uint64), ("members", ctypes.POINTER(MemberHP)),
                ("depth_lo", ctypes.c_int32), ("depth_hi", ctypes.c_int32),
                ("optimizer", ctypes.c_int32), ("ns_steps", ctypes.c_int32),
                ("muon_lr_lo", ctypes.c_double), ("muon_lr_hi", ctypes.c_double),
                ("muon_momentum", ctypes.c_double), ("muon_nesterov", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("emb_lo", ctypes.c_int32), ("emb_hi", ctypes.c_int32),
                ("emb_step", ctypes.c_int32), ("reserved3", ctypes.c_int32), ("sigma_lo", ctypes.c_double),
                ("sigma_hi", ctypes.c_double)]


class KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 64), ("kind", ctypes.c_int32), ("launches", ctypes.c_int32),
                ("total_ms", ctypes.c_double), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double), ("busy_ms", ctypes.c_double)]


class PackError(RuntimeError):
    pass


_LIB = None


def load_library(path=LIB_PATH):
    """Load libtabpack.so (once) and declare the C signatures."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise PackError(f"{path} is missing: build it first (python -m paper_2607_05380_amd.build)")
    L = ctypes.CDLL(path)
    vp, i32, i64, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t
    H = vp
    sig = {
        "pack_last_error": ([], ctypes.c_char_p),
        "pack_init": ([ctypes.POINTER(PackConfig), ctypes.POINTER(vp)], ctypes.c_int),
        "pack_destroy": ([H], ctypes.c_int),
        "pack_get_hparams": ([H, ctypes.POINTER(MemberHP)], ctypes.c_int),
        "pack_workspace_size": ([H, ctypes.POINTER(sz)], ctypes.c_int),
        "pack_bind": ([H, vp, sz, vp], ctypes.c_int),
        "pack_train_step": ([H, vp, vp, i64, vp, u64, vp, vp], ctypes.c_int),
        "pack_eval_members": ([H, vp, vp, i64, vp, vp, vp], ctypes.c_int),
        "pack_select_workspace_size": ([i32, i64, ctypes.POINTER(sz)], ctypes.c_int),
        "pack_select": ([H, vp, vp, i32, i64, i32, vp, sz, vp, vp, vp, vp], ctypes.c_int),
        "pack_select_static": ([H, vp, vp, i32, i64, i32, vp, vp, vp, vp], ctypes.c_int),
        "pack_member_param_count": ([H, i32, ctypes.POINTER(i64)], ctypes.c_int),
        "pack_get_params": ([H, i32, vp], ctypes.c_int),
        "pack_set_params": ([H, i32, vp], ctypes.c_int),
        "pack_get_grads": ([H, i32, vp], ctypes.c_int),
        "pack_get_moments": ([H, i32, vp, vp], ctypes.c_int),
        "pack_debug_dropout_mask": ([H, u64, i32, i32, vp, vp], ctypes.c_int),
        "pack_debug_activation": ([H, i32, i32, vp], ctypes.c_int),
        "pack_profile_enable": ([H, i32], ctypes.c_int),
        "pack_profile_read": ([H, ctypes.POINTER(KernelStat), i32, ctypes.POINTER(i32)], ctypes.c_int),
        "pack_set_active": ([H, vp, vp], ctypes.c_int),
        "pack_predict": ([H, vp, i64, i32, vp, vp], ctypes.c_int),
        "pack_status": ([H, ctypes.POINTER(ctypes.c_uint32), vp], ctypes.c_int),
        "pack_stream_copy": ([vp, vp, sz, vp], ctypes.c_int),
        "pack_bind_data": ([H, vp, i64, vp, sz, vp], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _LIB = L
    return L


def _check(rc):
    if rc != PACK_OK:
        raise PackError(f"tabpack error {rc}: {load_library().pack_last_error().decode()}")


def make_config(cfg, members=None):
    """PackConfig from a workload dict (see ``configs``; optional depth_lo/depth_hi
    give each member a depth drawn from that range); members: optional list of
    dicts {width, dropout, lr, wd[, depth]} overriding the sampled hyperparameters."""
    c = PackConfig()
    for f in ("K", "d_in", "d_out", "L", "B", "width_lo", "width_hi"):
        setattr(c, f, int(cfg.get(f, 0)))
    c.task = TASKS[cfg["task"]]
    c.precision = PRECISIONS[cfg.get("precision", "bf16")]
    c.quantum = int(cfg.get("quantum", 0))
    c.decay_bias = int(cfg.get("decay_bias", 1))
    c.keep_grads = int(cfg.get("keep_grads", 1))
    for f in ("dropout_lo", "dropout_hi", "lr_lo", "lr_hi", "wd_lo", "wd_hi"):
        setattr(c, f, float(cfg.get(f, 0.0)))
    c.beta1 = float(cfg.get("beta1", 0.9))
    c.beta2 = float(cfg.get("beta2", 0.999))
    c.eps = float(cfg.get("eps", 1e-8))
    c.seed = int(cfg["seed"])
    c.depth_lo = int(cfg.get("depth_lo", 0) or 0)
    c.depth_hi = int(cfg.get("depth_hi", 0) or 0)
    c.optimizer = OPTIMIZERS[cfg.get("optimizer", "adamw")]
    c.ns_steps = int(cfg.get("ns_steps", 5))
    c.muon_lr_lo = float(cfg.get("muon_lr_lo", 1e-3))
    c.muon_lr_hi = float(cfg.get("muon_lr_hi", 1e-1))
    c.muon_momentum = float(cfg.get("muon_momentum", 0.95))
    c.muon_nesterov = int(cfg.get("muon_nesterov", 1))
    c.emb_lo = int(cfg.get("emb_lo", 0) or 0)
    c.emb_hi = int(cfg.get("emb_hi", 0) or 0)
    c.emb_step = int(cfg.get("emb_step", 4) or 4)
    c.sigma_lo = float(cfg.get("sigma_lo", 1e-2))
    c.sigma_hi = float(cfg.get("sigma_hi", 10.0))
    keep = None
    if members is not None:
        keep = (MemberHP * len(members))()
        for i, m in enumerate(members):
            keep[i].width = int(m["width"])
            keep[i].dropout = float(m["dropout"])
            keep[i].lr = float(m["lr"])
            keep[i].wd = float(m["wd"])
            keep[i].depth = int(m.get("depth") or 0)
            keep[i].muon_lr = float(m.get("muon_lr", 0.0) or 0.0)
            keep[i].d_emb = int(m.get("d_emb", 0) or 0)
            keep[i].sigma = float(m.get("sigma", 0.0) or 0.0)
        c.members = ctypes.cast(keep, ctypes.POINTER(MemberHP))
    return c, keep


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class Pack:
    """A packed ensemble of K MLPs living in one library handle."""

    def __init__(self, cfg, members=None):
        self.lib = load_library()
        self.cfg = dict(cfg)
        c, keep = make_config(cfg, members)
        h = ctypes.c_void_p()
        _check(self.lib.pack_init(ctypes.byref(c), ctypes.byref(h)))
        del keep
        self.h = h
        self.K, self.L, self.B = c.K, c.L, c.B
        self.d_in, self.d_out = c.d_in, c.d_out
        self.workspace = None
        self._select_ws = None
        self.xb = None
        self.active = [True] * self.K

    def __del__(self):
        h = getattr(self, "h", None)
        if h is not None and h.value:
            self.lib.pack_destroy(h)
            self.h = None

    # ------------------------------------------------------------ set-up
    def hparams(self):
        arr = (MemberHP * self.K)()
        _check(self.lib.pack_get_hparams(self.h, arr))
        return [dict(width=a.width, padded_width=a.padded_width, t=a.drop_threshold, depth=a.depth,
                     dropout=a.dropout, lr=a.lr, wd=a.wd, s=a.scale, muon_lr=a.muon_lr, d_emb=a.d_emb,
                     sigma=a.sigma) for a in arr]

    def workspace_bytes(self):
        n = ctypes.c_size_t()
        _check(self.lib.pack_workspace_size(self.h, ctypes.byref(n)))
        return n.value

    def bind(self, device="cuda"):
        import torch
        self.workspace = torch.empty(self.workspace_bytes(), dtype=torch.uint8, device=device)
        _check(self.lib.pack_bind(self.h, ctypes.c_void_p(self.workspace.data_ptr()),
                                  self.workspace.numel(), _stream()))
        return self

    # ------------------------------------------------------------ hot path
    def train_step(self, X, y, idx, step, loss_out=None):
        """X fp32 [N, d_in], y fp32/int32 [N], idx int32 [K, B] (device tensors)."""
        import torch
        assert X.is_cuda and X.dtype == torch.float32 and X.is_contiguous() and X.shape[1] == self.d_in
        assert idx.dtype == torch.int32 and idx.is_contiguous() and tuple(idx.shape) == (self.K, self.B)
        assert y.is_contiguous() and y.shape[0] == X.shape[0]
        if loss_out is None:
            loss_out = torch.empty(self.K, dtype=torch.float32, device=X.device)
        _check(self.lib.pack_train_step(self.h, X.data_ptr(), y.data_ptr(), X.shape[0], idx.data_ptr(),
                                        int(step), loss_out.data_ptr(), _stream()))
        return loss_out

    def can_bind_data(self):
        """Whether bind_data applies: bf16 packs without feature embeddings and
        with B <= BIND_DATA_MAX_B."""
        c = self.cfg
        return (c.get("precision", "bf16") == "bf16" and int(c.get("emb_lo", 0) or 0) == 0
                and self.B <= BIND_DATA_MAX_B)

    def bind_data(self, X):
        """Let the first layer's forward and weight-gradient GEMMs read the batch
        rows straight from X (device fp32 [N, d_in]) through the batch indices,
        with no gathered copy of the batch; every later train_step must pass
        this X.  bind_data(None) unbinds.  Keeps the bf16 copy of X it makes."""
        import torch
        if X is None:
            _check(self.lib.pack_bind_data(self.h, None, 0, None, 0, _stream()))
            self.xb = None
            return self
        assert X.is_cuda and X.dtype == torch.float32 and X.is_contiguous() and X.shape[1] == self.d_in
        pin = (self.d_in + 7) // 8 * 8
        xb = torch.empty(X.shape[0] * pin, dtype=torch.bfloat16, device=X.device)
        _check(self.lib.pack_bind_data(self.h, X.data_ptr(), X.shape[0], xb.data_ptr(), xb.numel() * 2, _stream()))
        self.xb = xb
        return self

    def status(self):
        """Asynchronous error flags raised since the last call (waits for the
        current stream, then clears them): STATUS_IDX_RANGE when a batch index
        lay outside [0, N)."""
        flags = ctypes.c_uint32()
        _check(self.lib.pack_status(self.h, ctypes.byref(flags), _stream()))
        return flags.value

    def set_active(self, active, stream=None):
        """active: K booleans; removed members are frozen and leave the launches."""
        assert len(active) == self.K
        arr = (ctypes.c_uint8 * self.K)(*[1 if a else 0 for a in active])
        _check(self.lib.pack_set_active(self.h, arr, _stream(stream)))
        self.active = [bool(a) for a in active]

    def eval_members(self, Xv, yv):
        """(pred fp32 [K, Nv], score fp64 [K]); rows of inactive members are NaN."""
        import torch
        assert Xv.is_cuda and Xv.dtype == torch.float32 and Xv.is_contiguous() and Xv.shape[1] == self.d_in
        Nv = Xv.shape[0]
        pred = torch.full((self.K, Nv), float("nan"), dtype=torch.float32, device=Xv.device)
        score = torch.full((self.K,), float("nan"), dtype=torch.float64, device=Xv.device)
        _check(self.lib.pack_eval_members(self.h, Xv.data_ptr(), yv.data_ptr(), Nv, pred.data_ptr(),
                                          score.data_ptr(), _stream()))
        return pred, score

    def predict(self, X, ensemble=False):
        """Predictions without dropout: [n_active, N, d_out] per active member (increasing
        index), or the ensemble mean [N, d_out] with ensemble=True."""
        import torch
        assert X.is_cuda and X.dtype == torch.float32 and X.is_contiguous() and X.shape[1] == self.d_in
        N = X.shape[0]
        shape = (N, self.d_out) if ensemble else (sum(self.active), N, self.d_out)
        out = torch.empty(shape, dtype=torch.float32, device=X.device)
        _check(self.lib.pack_predict(self.h, X.data_ptr(), N, PREDICT_ENSEMBLE if ensemble else PREDICT_MEMBERS,
                                     out.data_ptr(), _stream()))
        return out

    def select(self, cand, yv, m_ens):
        """Greedy selection over cand fp32 [C, Nv]; returns (picks, score) on the host."""
        import torch
        C, Nv = cand.shape
        n = ctypes.c_size_t()
        _check(self.lib.pack_select_workspace_size(C, Nv, ctypes.byref(n)))
        if self._select_ws is None or self._select_ws.numel() < n.value:
            self._select_ws = torch.empty(n.value, dtype=torch.uint8, device=cand.device)
        sel = torch.full((max(m_ens, 1),), -1, dtype=torch.int32, device=cand.device)
        nsel = torch.zeros(1, dtype=torch.int32, device=cand.device)
        score = torch.zeros(1, dtype=torch.float64, device=cand.device)
        _check(self.lib.pack_select(self.h, cand.data_ptr(), yv.data_ptr(), C, Nv, m_ens,
                                    self._select_ws.data_ptr(), self._select_ws.numel(), sel.data_ptr(),
                                    nsel.data_ptr(), score.data_ptr(), _stream()))
        torch.cuda.current_stream().synchronize()
        k = int(nsel.item())
        return [int(x) for x in sel[:k].cpu()], float(score.item())

    def select_static(self, cand, yv, m_ens, sel, nsel, score):
        """pack_select_static: the selection of ``select`` into caller-provided
        device outputs (sel int32 [>= max(m_ens, 1)], nsel int32 [1], score fp64
        [1]) with the library's static scratch, on the current stream: no
        allocation and no synchronisation."""
        C, Nv = cand.shape
        _check(self.lib.pack_select_static(self.h, cand.data_ptr(), yv.data_ptr(), C, Nv, m_ens, sel.data_ptr(),
                                           nsel.data_ptr(), score.data_ptr(), _stream()))

    # ------------------------------------------------------------ state access
    def param_count(self, k):
        n = ctypes.c_int64()
        _check(self.lib.pack_member_param_count(self.h, k, ctypes.byref(n)))
        return n.value

    def _dense(self, fn, k):
        out = np.empty(self.param_count(k), dtype=np.float32)
        _check(fn(self.h, k, out.ctypes.data))
        return out

    def get_params(self, k):
        return self.split(k, self._dense(self.lib.pack_get_params, k))

    def get_grads(self, k):
        return self.split(k, self._dense(self.lib.pack_get_grads, k))

    def get_moments(self, k):
        n = self.param_count(k)
        m = np.empty(n, dtype=np.float32)
        v = np.empty(n, dtype=np.float32)
        _check(self.lib.pack_get_moments(self.h, k, m.ctypes.data, v.ctypes.data))
        return self.split(k, m), self.split(k, v)

    def set_params(self, k, params):
        """params as ``split`` returns them (embedding dict first when the pack has embeddings)."""
        parts = []
        for p in params:
            if isinstance(p, dict):
                parts += [np.asarray(p[n], np.float32).ravel() for n in ("w", "b", "alpha", "beta")]
            else:
                parts += [np.asarray(p[0], np.float32).ravel(), np.asarray(p[1], np.float32).ravel()]
        flat = np.concatenate(parts)
        assert flat.size == self.param_count(k)
        flat = np.ascontiguousarray(flat)
        _check(self.lib.pack_set_params(self.h, k, flat.ctypes.data))

    def split(self, k, flat):
        """Dense member vector -> [(W [out, in], b [out]), ...] for the L_k blocks and the head,
        preceded by a dict of the embedding parameters w, b [d_in, d_emb-1], alpha, beta
        [d_in, d_emb] when the pack has embeddings."""
        hp = self.hparams()[k]
        w, depth, de = hp["width"], hp["depth"], hp["d_emb"]
        dims = [self.d_in * de if de else self.d_in] + [w] * depth + [self.d_out]
        out, o = [], 0
        if de:
            emb = {}
            for n, cols in (("w", de - 1), ("b", de - 1), ("alpha", de), ("beta", de)):
                emb[n] = flat[o:o + self.d_in * cols].reshape(self.d_in, cols)
                o += self.d_in * cols
            out.append(emb)
        for i in range(depth + 1):
            n_in, n_out = dims[i], dims[i + 1]
            W = flat[o:o + n_in * n_out].reshape(n_out, n_in)
            o += n_in * n_out
            b = flat[o:o + n_out]
            o += n_out
            out.append((W, b))
        return out

    def debug_dropout_mask(self, step, layer, k):
        import torch
        w = self.hparams()[k]["width"]
        out = torch.empty((self.B, w), dtype=torch.uint8, device="cuda")
        _check(self.lib.pack_debug_dropout_mask(self.h, int(step), layer, k, out.data_ptr(), _stream()))
        torch.cuda.current_stream().synchronize()
        return out.cpu().numpy().astype(bool)

    def profile(self, enable):
        _check(self.lib.pack_profile_enable(self.h, 1 if enable else 0))

    def profile_read(self):
        """[{name, kind ('mfma'|'hbm'), launches, total_ms, avg_ms, busy_ms, flops, bytes (per launch)}]"""
        arr = (KernelStat * 64)()
        n = ctypes.c_int32()
        _check(self.lib.pack_profile_read(self.h, arr, 64, ctypes.byref(n)))
        out = []
        for s in arr[:n.value]:
            out.append(dict(name=s.name.decode(), kind="mfma" if s.kind == 0 else "hbm", launches=s.launches,
                            total_ms=s.total_ms, avg_ms=s.total_ms / max(s.launches, 1), busy_ms=s.busy_ms,
                            flops=s.flops, bytes=s.bytes))
        return out

    def debug_activation(self, layer, k):
        w = self.hparams()[k]["width"]
        out = np.empty((self.B, w), dtype=np.float32)
        _check(self.lib.pack_debug_activation(self.h, layer, k, out.ctypes.data))
        return out


def stream_copy(src, dst):
    """dst <- src (device tensors of equal byte size, 16-byte multiples) with the
    library's non-temporal streaming kernel, on the current stream."""
    n = src.numel() * src.element_size()
    assert src.is_cuda and dst.is_cuda and dst.numel() * dst.element_size() == n
    _check(load_library().pack_stream_copy(src.data_ptr(), dst.data_ptr(), n, _stream()))
