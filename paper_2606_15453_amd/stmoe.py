"""Python binding of libstmoe.so (ctypes).

Argument marshalling only: torch tensors become raw device/host pointers,
torch streams become hipStream_t handles, and every call goes straight to
the C ABI declared in include/stmoe.h.  Nothing here computes any step of
the decode-step MoE layer.  Importing this module loads the library and
raises if it has not been built (see paper_2606_15453_amd.build).
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libstmoe.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_15453_amd.build`")

# torch must load its HIP runtime first: the library then binds to that same
# runtime (matching SONAME) instead of mapping a second one into the process.
import torch  # noqa: E402,F401

_lib = C.CDLL(LIB_PATH)


def _hip_runtimes():
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            if "libamdhip64" in line:
                paths.add(line.split()[-1])
    return sorted(paths)


if len(_hip_runtimes()) > 1:
    raise ImportError(f"more than one HIP runtime mapped: {_hip_runtimes()}")

OK, EINVAL, EHIP, ENOMEM, ECAPACITY, ESTATE = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
USE_CCT, USE_HT, USE_BOTH = 1, 2, 3
MODE_ON_DEMAND, MODE_STMOE, MODE_HT_ONLY, MODE_CCT_ONLY = 0, 1, 2, 3

vp, i32, i64, sz = C.c_void_p, C.c_int, C.c_int64, C.c_size_t
P = C.POINTER


class CacheStats(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("hits", "demand", "overflow", "prefetch", "useful", "wasted")]

    def as_dict(self):
        return {n: int(getattr(self, n)) for n, _ in self._fields_}


class LayerReport(C.Structure):
    _fields_ = [("B", i32), ("K", i32), ("idx", i32 * 256), ("w", C.c_float * 256),
                ("n_ranked", i32), ("ranked", i32 * 256), ("pred_stats", i64 * 3),
                ("cache", CacheStats)]

    def as_dict(self):
        bk = self.B * self.K
        n = self.n_ranked
        return dict(idx=np.array(self.idx[:bk], np.int32).reshape(self.B, self.K),
                    w=np.array(self.w[:bk], np.float32).reshape(self.B, self.K),
                    n_ranked=n, ranked=list(self.ranked[:max(n, 0)]),
                    pred_stats=tuple(self.pred_stats), cache=self.cache.as_dict())


class ModelDesc(C.Structure):
    _fields_ = [("L", i32), ("E", i32), ("K", i32), ("B", i32), ("H", i32), ("I", i32),
                ("n_shared", i32), ("dtype", i32), ("renorm", i32),
                ("router_w", P(vp)), ("shared_w", P(vp)), ("resident_w", P(vp))]


_SIGS = {
    "stmoe_last_error": (C.c_char_p, []),
    "stmoe_abi_version": (i32, []),
    "stmoe_host_alloc": (i32, [sz, P(vp)]),
    "stmoe_host_free": (i32, [vp]),
    "moe_route_workspace_bytes": (sz, [i32, i32]),
    "moe_route_topk": (i32, [vp, vp, i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, sz, vp]),
    "stmoe_workspace_bytes": (sz, [i32, i32, i32, i32]),
    "stmoe_create": (i32, [i32, i32, i32, i32, vp, sz, P(vp)]),
    "stmoe_destroy": (i32, [vp]),
    "stmoe_profile": (i32, [vp, vp, i32]),
    "stmoe_update": (i32, [vp, i32, vp, vp, i32, vp]),
    "stmoe_predict": (i32, [vp, i32, vp, i32, vp, vp, vp, vp, vp, vp]),
    "stmoe_export": (i32, [vp, vp, vp, vp, vp]),
    "stmoe_import": (i32, [vp, vp, vp, vp]),
    "stmoe_stats": (i32, [vp, vp]),
    "moe_blob_bytes": (sz, [i32, i32, i32]),
    "moe_pack_expert": (i32, [vp, vp, vp, i32, i32, i32, vp]),
    "moe_expert_ffn_workspace_bytes": (sz, [i32, i32, i32, i32, i32, i32, i32]),
    "moe_expert_ffn": (i32, [vp, vp, vp, i32, i32, i32, i32, i32, i32, vp, vp, i32, vp, vp, sz, vp]),
    "moe_expert_ffn_noalloc": (i32, [vp, vp, vp, i32, i32, i32, i32, i32, i32, vp, vp, i32, vp, vp]),
    "expert_cache_warm_sets": (i32, [vp, i32, i32, i32, i32, i32, i32, vp]),
    "expert_cache_use_counts": (i32, [vp, i32, i32, i32, i32, i32, vp]),
    "stmoe_policy_set_counts": (i32, [vp, vp]),
    "expert_cache_set_counts": (i32, [vp, vp]),
    "stmoe_policy_create": (i32, [i32, i32, i32, vp, P(vp)]),
    "stmoe_policy_destroy": (i32, [vp]),
    "stmoe_policy_prefetch": (i32, [vp, i32, vp, i32, i64, vp]),
    "stmoe_policy_acquire": (i32, [vp, i32, vp, i32, i64, vp, vp]),
    "stmoe_policy_slots": (i32, [vp, vp]),
    "stmoe_policy_stats": (i32, [vp, P(CacheStats)]),
    "expert_cache_arena_bytes": (sz, [i32, i32, i32, sz, i32]),
    "expert_cache_create": (i32, [i32, i32, i32, sz, i32, vp, sz, P(vp), vp, vp, P(vp)]),
    "expert_cache_destroy": (i32, [vp]),
    "expert_cache_warm": (i32, [vp, vp]),
    "expert_cache_prefetch": (i32, [vp, i32, vp, i32, i64]),
    "expert_cache_acquire": (i32, [vp, i32, vp, i32, i64, P(vp), vp]),
    "expert_cache_release": (i32, [vp, i32, vp]),
    "expert_cache_set_prefetch_order": (i32, [vp, i32]),
    "expert_cache_set_device_policy": (i32, [vp, i32]),
    "expert_cache_set_staged_prefetch": (i32, [vp, i32, sz]),
    "expert_cache_stats": (i32, [vp, P(CacheStats)]),
    "moe_ctx_workspace_bytes": (sz, [P(ModelDesc)]),
    "moe_ctx_create": (i32, [P(ModelDesc), vp, vp, vp, vp, sz, P(vp)]),
    "moe_ctx_destroy": (i32, [vp]),
    "moe_decode_layer": (i32, [vp, i32, i32, vp, vp, i32, P(LayerReport)]),
    "moe_decode_token": (i32, [vp, i32, vp, vp, i32]),
    "moe_ctx_set_prefetch": (i32, [vp, i32, i32]),
    "moe_ctx_set_online_update": (i32, [vp, i32]),
    "moe_ctx_set_predictor_batch": (i32, [vp, i32]),
    "moe_ctx_last_routing": (i32, [vp, vp, vp]),
    "moe_ctx_set_timing": (i32, [vp, i32]),
    "moe_ctx_set_graph": (i32, [vp, i32]),
    "moe_ctx_graph_buffers": (i32, [vp, P(vp), P(vp)]),
    "moe_ctx_timing": (i32, [vp, P(C.c_double), P(C.c_double), P(i64), P(i64)]),
    "moe_ctx_stage_timing": (i32, [vp, P(C.c_double), P(C.c_double), P(C.c_double), P(C.c_double), P(i64)]),
    "stmoe_calib_copy": (i32, [vp, vp, sz, vp]),
    "stmoe_calib_read_out_words": (sz, [sz, i32]),
    "stmoe_calib_copy_grid": (i32, [vp, vp, sz, i32, vp]),
    "expert_cache_set_copy_workgroups": (i32, [vp, i32, i32]),
    "stmoe_calib_read": (i32, [vp, sz, i32, vp, vp]),
    "stmoe_calib_handoff": (i32, [vp, sz, i32, vp, sz, i32, i32, vp, vp, vp, C.c_uint, vp]),
}

for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = tuple(_SIGS)


class StmoeError(RuntimeError):
    def __init__(self, fn, rc):
        msg = _lib.stmoe_last_error().decode()
        super().__init__(f"{fn} failed with status {rc}: {msg}")
        self.rc = rc


def _call(name, *args):
    rc = getattr(_lib, name)(*args)
    if rc < 0:
        raise StmoeError(name, rc)
    return rc


def _p(t):
    """Raw pointer of a torch tensor / numpy array / int / None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _s(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def abi_version() -> int:
    return _lib.stmoe_abi_version()


def device_workspace(nbytes, device="cuda:0"):
    """A zeroed device buffer of at least `nbytes` whose returned address is
    256-byte aligned: (tensor keeping it alive, aligned address)."""
    t = torch.zeros(int(nbytes) + 256, dtype=torch.uint8, device=device)
    return t, (t.data_ptr() + 255) // 256 * 256


class PinnedHost:
    """A pinned host block of exactly `nbytes` (stmoe_host_alloc), viewable as a
    CPU uint8 tensor; freed on close()."""

    def __init__(self, nbytes):
        p = vp()
        _call("stmoe_host_alloc", nbytes, C.byref(p))
        self.ptr, self.nbytes = p.value, nbytes

    def tensor(self, offset=0, nbytes=None):
        n = self.nbytes - offset if nbytes is None else nbytes
        buf = (C.c_uint8 * n).from_address(self.ptr + offset)
        return torch.frombuffer(buf, dtype=torch.uint8)

    def close(self):
        if self.ptr:
            _lib.stmoe_host_free(self.ptr)
            self.ptr = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- gating
def route_workspace_bytes(B, E):
    return _lib.moe_route_workspace_bytes(B, E)


def route_topk(x, w_gate, K, idx, w, ws, renorm=False, logits=None, stream=None, dtype=None):
    B, H = x.shape
    E = w_gate.shape[0]
    dt = dtype if dtype is not None else (BF16 if x.element_size() == 2 else F32)
    _call("moe_route_topk", _p(x), _p(w_gate), B, H, E, K, dt, int(renorm), _p(idx), _p(w),
          _p(logits), _p(ws), ws.numel() * ws.element_size(), _s(stream))


# ------------------------------------------------------------- predictor
def predictor_workspace_bytes(L, E, K, B):
    return _lib.stmoe_workspace_bytes(L, E, K, B)


class Predictor:
    """stmoe_predictor over a device workspace this object allocates (torch)."""

    def __init__(self, L, E, K, B):
        self.L, self.E, self.K, self.B = L, E, K, B
        nbytes = _lib.stmoe_workspace_bytes(L, E, K, B)
        if nbytes == 0:
            raise StmoeError("stmoe_workspace_bytes", EINVAL)
        self._ws, ptr = device_workspace(nbytes)
        h = vp()
        _call("stmoe_create", L, E, K, B, ptr, nbytes, C.byref(h))
        self.h = h

    def close(self):
        if self.h:
            _lib.stmoe_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def profile(self, sel):
        sel = _i32(sel)
        _call("stmoe_profile", self.h, sel.ctypes.data, sel.shape[0])

    def update(self, layer, sel_prev, sel_cur, online=True, stream=None):
        _call("stmoe_update", self.h, layer, _p(sel_prev), _p(sel_cur), int(online), _s(stream))

    def predict(self, layer, sel_cur, use=USE_BOTH, score=None, mask=None, ranked=None,
                n_ranked=None, max_score=None, stream=None):
        _call("stmoe_predict", self.h, layer, _p(sel_cur), use, _p(score), _p(mask), _p(max_score),
              _p(ranked), _p(n_ranked), _s(stream))

    def export(self):
        L, E, K, B = self.L, self.E, self.K, self.B
        pr = max(L - 1, 0)
        co = np.zeros((pr, E, E), np.int32)
        ci = np.zeros((pr, E, K), np.uint8)
        cc = np.zeros((pr, E, K), np.uint8)
        ht = np.zeros((L, B, K), np.int32)
        _call("stmoe_export", self.h, co.ctypes.data, ci.ctypes.data, cc.ctypes.data, ht.ctypes.data)
        return co, ci, cc, ht

    def import_tables(self, cct_idx, cct_conf, ht):
        ci = np.ascontiguousarray(cct_idx, np.uint8)
        cc = np.ascontiguousarray(cct_conf, np.uint8)
        h = np.ascontiguousarray(ht, np.int32)
        _call("stmoe_import", self.h, ci.ctypes.data, cc.ctypes.data, h.ctypes.data)

    def stats(self):
        out = np.zeros((self.L, 3), np.int64)
        _call("stmoe_stats", self.h, out.ctypes.data)
        return out


# ------------------------------------------------------------- packing
def blob_bytes(H, I, dtype):
    return _lib.moe_blob_bytes(H, I, dtype)


def pack_expert(w_gate, w_up, w_down, dtype, out):
    I, H = w_gate.shape
    _call("moe_pack_expert", _p(w_gate), _p(w_up), _p(w_down), H, I, dtype, _p(out))


# ------------------------------------------------------------- FFN
def ffn_workspace_bytes(B, K, E, H, I, n_shared=0, dtype=BF16):
    """Workspace bytes for expert_ffn; allocate zero-filled (torch.zeros), 256-byte aligned."""
    return _lib.moe_expert_ffn_workspace_bytes(B, K, E, H, I, n_shared, dtype)


def expert_ffn(x, idx, w, H, I, E, dtype, expert_ptrs, y, ws, shared_ptrs=None, n_shared=0,
               stream=None):
    B, K = idx.shape
    _call("moe_expert_ffn", _p(x), _p(idx), _p(w), B, K, H, I, E, dtype, _p(expert_ptrs),
          _p(shared_ptrs), n_shared, _p(y), _p(ws), ws.numel() * ws.element_size(), _s(stream))


def expert_ffn_noalloc(x, idx, w, H, I, E, dtype, expert_ptrs, y, shared_ptrs=None, n_shared=0,
                       stream=None):
    """moe_expert_ffn_noalloc: the expert FFN on the library's per-GPU scratch (no workspace)."""
    B, K = idx.shape
    _call("moe_expert_ffn_noalloc", _p(x), _p(idx), _p(w), B, K, H, I, E, dtype, _p(expert_ptrs),
          _p(shared_ptrs), n_shared, _p(y), _s(stream))


# ------------------------------------------------------------- cache policy
def warm_sets(sel, E, C_):
    """expert_cache_warm_sets: per layer the C most-profiled experts ([L][C], -1 padding)."""
    sel = _i32(sel)
    P_, B_, L_, K_ = sel.shape
    out = np.zeros((L_, C_), np.int32)
    _call("expert_cache_warm_sets", sel.ctypes.data, P_, B_, L_, K_, E, C_, out.ctypes.data)
    return out


def use_counts(sel, E):
    """expert_cache_use_counts: per layer, profiling tokens selecting each expert ([L][E] int64)."""
    sel = _i32(sel)
    P_, B_, L_, K_ = sel.shape
    out = np.zeros((L_, E), np.int64)
    _call("expert_cache_use_counts", sel.ctypes.data, P_, B_, L_, K_, E, out.ctypes.data)
    return out


def _counts_ptr(counts):
    if counts is None:
        return None, None
    a = np.ascontiguousarray(counts, np.int64)
    return a, a.ctypes.data


class Policy:
    def __init__(self, L, E, C_, warm=None):
        self.L, self.E, self.C = L, E, C_
        h = vp()
        wa = None if warm is None else _i32(warm)
        _call("stmoe_policy_create", L, E, C_, None if wa is None else wa.ctypes.data, C.byref(h))
        self.h = h

    def __del__(self):
        if getattr(self, "h", None):
            _lib.stmoe_policy_destroy(self.h)
            self.h = None

    def prefetch(self, layer, ranked, stamp):
        r = _i32(ranked)
        pairs = np.zeros(2 * self.C + 2, np.int32)
        n = _call("stmoe_policy_prefetch", self.h, layer, r.ctypes.data, len(r), stamp, pairs.ctypes.data)
        return [tuple(pairs[2 * i:2 * i + 2].tolist()) for i in range(n)]

    def acquire(self, layer, needed, stamp):
        r = _i32(needed)
        pairs = np.zeros(2 * max(len(r), 1), np.int32)
        nh = C.c_int32()
        n = _call("stmoe_policy_acquire", self.h, layer, r.ctypes.data, len(r), stamp, pairs.ctypes.data,
                  C.byref(nh))
        return [tuple(pairs[2 * i:2 * i + 2].tolist()) for i in range(n)], nh.value

    def slots(self):
        out = np.zeros((self.L, self.C), np.int32)
        _call("stmoe_policy_slots", self.h, out.ctypes.data)
        return out

    def set_counts(self, counts):
        keep, ptr = _counts_ptr(counts)
        _call("stmoe_policy_set_counts", self.h, ptr)

    def stats(self):
        st = CacheStats()
        _call("stmoe_policy_stats", self.h, C.byref(st))
        return st.as_dict()


# ------------------------------------------------------------- HBM cache
def cache_arena_bytes(L, E, C_, blob, n_stage):
    return _lib.expert_cache_arena_bytes(L, E, C_, blob, n_stage)


class ExpertCache:
    def __init__(self, L, E, C_, blob, n_stage, arena, host_ptrs, demand_stream, side_stream):
        self.L, self.E, self.C = L, E, C_
        self._host = (vp * (L * E))(*[int(p) for p in host_ptrs])
        h = vp()
        _call("expert_cache_create", L, E, C_, blob, n_stage, _p(arena), arena.numel() * arena.element_size(),
              self._host, _s(demand_stream), _s(side_stream), C.byref(h))
        self.h = h
        self._arena = arena

    def close(self):
        if self.h:
            _lib.expert_cache_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def warm(self, warm):
        w = _i32(warm)
        _call("expert_cache_warm", self.h, w.ctypes.data)

    def prefetch(self, layer, ranked, stamp):
        r = _i32(ranked)
        return _call("expert_cache_prefetch", self.h, layer, r.ctypes.data, len(r), stamp)

    def acquire(self, layer, needed, stamp, compute_stream=None):
        r = _i32(needed)
        tab = (vp * self.E)()
        hits = _call("expert_cache_acquire", self.h, layer, r.ctypes.data, len(r), stamp, tab,
                     _s(compute_stream))
        return hits, [tab[e] for e in range(self.E)]

    def release(self, layer, compute_stream=None):
        _call("expert_cache_release", self.h, layer, _s(compute_stream))

    def set_prefetch_order(self, after_demand):
        _call("expert_cache_set_prefetch_order", self.h, int(after_demand))

    def set_device_policy(self, on):
        _call("expert_cache_set_device_policy", self.h, int(on))

    def set_copy_workgroups(self, demand=0, prefetch=0):
        """Copy-kernel workgroups with device decisions (0: defaults)."""
        _call("expert_cache_set_copy_workgroups", self.h, int(demand), int(prefetch))

    def set_counts(self, counts):
        """Frequency-aware eviction seeded with counts [L][E], or least recently used (None)."""
        keep, ptr = _counts_ptr(counts)
        _call("expert_cache_set_counts", self.h, ptr)

    def set_staged_prefetch(self, n_per_layer, head_bytes=0):
        """Prefetch into spare staging blocks (at most n per layer); unused ones are cancelled
        (device decisions) or stop after their first head_bytes (host decisions)."""
        _call("expert_cache_set_staged_prefetch", self.h, int(n_per_layer), int(head_bytes))

    def stats(self):
        st = CacheStats()
        _call("expert_cache_stats", self.h, C.byref(st))
        return st.as_dict()


# ------------------------------------------------------------- decode layer
class DecodeContext:
    """moe_ctx: one MoE decode stack on one stream (router, predictor, cache/FFN)."""

    def __init__(self, L, E, K, B, H, I, dtype, router_ptrs, predictor=None, cache=None,
                 resident_ptrs=None, shared_ptrs=None, n_shared=0, renorm=False, stream=None):
        self.L, self.E, self.K, self.B = L, E, K, B
        self._router = (vp * L)(*[int(p) for p in router_ptrs])
        self._resident = None if resident_ptrs is None else (vp * (L * E))(*[int(p) for p in resident_ptrs])
        self._shared = None if not n_shared else (vp * (L * n_shared))(*[int(p) for p in shared_ptrs])
        d = ModelDesc(L, E, K, B, H, I, n_shared, dtype, int(renorm), self._router,
                      self._shared, self._resident)
        nbytes = _lib.moe_ctx_workspace_bytes(C.byref(d))
        if nbytes == 0:
            raise StmoeError("moe_ctx_workspace_bytes", EINVAL)
        self._ws, ptr = device_workspace(nbytes)
        h = vp()
        _call("moe_ctx_create", C.byref(d), predictor.h if predictor else None,
              cache.h if cache else None, _s(stream), ptr, nbytes, C.byref(h))
        self.h = h
        self._keep = (predictor, cache)

    def close(self):
        if self.h:
            _lib.moe_ctx_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def layer(self, token, layer, x, y, mode=MODE_STMOE, report=False):
        """One layer; with report=True waits for it and returns its moe_layer_report as a dict."""
        rep = LayerReport() if report else None
        _call("moe_decode_layer", self.h, token, layer, _p(x), _p(y), mode,
              C.byref(rep) if report else None)
        return rep.as_dict() if report else None

    def set_prefetch(self, min_score=2, max_per_layer=1 << 30):
        _call("moe_ctx_set_prefetch", self.h, min_score, max_per_layer)

    def set_online_update(self, on=True):
        """Algorithm 3's CCT update during decode on, or the CCTs frozen after profiling."""
        _call("moe_ctx_set_online_update", self.h, int(bool(on)))

    def token(self, token, xs, ys, mode=MODE_STMOE):
        _call("moe_decode_token", self.h, token, _p(xs), _p(ys), mode)

    def last_routing(self):
        idx = np.zeros((self.L, self.B, self.K), np.int32)
        w = np.zeros((self.L, self.B, self.K), np.float32)
        _call("moe_ctx_last_routing", self.h, idx.ctypes.data, w.ctypes.data)
        return idx, w

    def set_timing(self, every):
        """Time the FFN of every `every`-th token (0 stops; True means every token)."""
        _call("moe_ctx_set_timing", self.h, int(every))

    def set_predictor_batch(self, on=True):
        """One side-stream predictor launch per token (every layer's update and
        prediction, in order) instead of one per layer; contexts without a cache."""
        _call("moe_ctx_set_predictor_batch", self.h, int(bool(on)))

    def set_graph(self, on=True):
        """Replay each token (after the first) as one HIP graph; no-cache contexts only."""
        _call("moe_ctx_set_graph", self.h, int(bool(on)))

    def graph_buffers(self):
        """(x_stage, y_stage) device addresses of the graph's staging buffers."""
        x, y = vp(), vp()
        _call("moe_ctx_graph_buffers", self.h, C.byref(x), C.byref(y))
        return x.value, y.value

    def timing(self):
        """(gate/up kernel ms, down kernel ms, FFN calls, distinct routed experts) since set_timing(1)."""
        up, down = C.c_double(), C.c_double()
        nc, ne = i64(), i64()
        _call("moe_ctx_timing", self.h, C.byref(up), C.byref(down), C.byref(nc), C.byref(ne))
        return up.value, down.value, nc.value, ne.value

    def stage_timing(self):
        """(route ms, miss ms, FFN ms, side-stream predict ms, timed layers) since set_timing(every)."""
        r, m, f, p = C.c_double(), C.c_double(), C.c_double(), C.c_double()
        n = i64()
        _call("moe_ctx_stage_timing", self.h, C.byref(r), C.byref(m), C.byref(f), C.byref(p), C.byref(n))
        return r.value, m.value, f.value, p.value, n.value


# ------------------------------------------------------------- measurement
def calib_copy(src, dst, nbytes, stream=None):
    _call("stmoe_calib_copy", _p(src), _p(dst), nbytes, _s(stream))


def calib_read(src, nbytes, out, stream=None, pattern=0):
    """Streaming read of nbytes: pattern 0 grid stride, 1 contiguous 256 KiB per workgroup."""
    _call("stmoe_calib_read", _p(src), nbytes, int(pattern), _p(out), _s(stream))


def calib_copy_grid(src_ptr, dst_ptr, nbytes, workgroups, stream=None):
    """stmoe_calib_copy_grid between raw device-accessible addresses."""
    _call("stmoe_calib_copy_grid", src_ptr, dst_ptr, nbytes, int(workgroups), _s(stream))


def calib_read_out_words(nbytes, pattern=0):
    return _lib.stmoe_calib_read_out_words(nbytes, int(pattern))


HANDOFF_SYNC_WORDS = 64 + 64 * 1024   # sync words modes 3 and 4 of stmoe_calib_handoff use


def calib_handoff(w1, chunk1, producers, w2, chunk2, consumers, mode, act, out, sync, target, stream=None):
    """stmoe_calib_handoff: producers publish one word each, consumers read them
    all (mode 0 two launches, 1-4 one launch with an in-kernel wait; modes 3
    and 4 need HANDOFF_SYNC_WORDS words of sync)."""
    if mode >= 3 and sync.numel() * sync.element_size() < 4 * HANDOFF_SYNC_WORDS:
        raise ValueError("modes 3 and 4 need HANDOFF_SYNC_WORDS words of sync")
    _call("stmoe_calib_handoff", _p(w1), chunk1, int(producers), _p(w2), chunk2, int(consumers), int(mode),
          _p(act), _p(out), _p(sync), int(target) & 0xFFFFFFFF, _s(stream))
