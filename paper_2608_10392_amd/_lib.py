"""ctypes binding of libunifmoe.so (include/unif_moe.h).

Argument marshalling only: every step of the layer runs in the HIP library.
Tensors are torch device tensors (torch provides device memory and streams);
the library never falls back to anything else, and loading fails loudly when
the built library is missing.
"""
import ctypes
import math
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libunifmoe.so")

OK, EINVAL, EWORKSPACE, EDEVICE, EUNSUPPORTED, ECAPACITY = 0, -1, -2, -3, -4, -5
DTYPES = {"f32": 0, "bf16": 1}
ALPHA_MODES = {"adaptive": 0, "fixed": 1}
MASS_MODES = {"coupled": 0, "fixed": 1, "topk": 2}
SELECT_MODES = {"prototype": 0, "prefix": 1}


class Config(ctypes.Structure):
    _fields_ = [("n_tokens", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("n_blocks", ctypes.c_int32),
                ("block_width", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("tau", ctypes.c_float), ("mass_threshold", ctypes.c_float),
                ("max_shared", ctypes.c_int32), ("alpha_mode", ctypes.c_int32),
                ("alpha_fixed", ctypes.c_float), ("mass_mode", ctypes.c_int32),
                ("fixed_k", ctypes.c_int32), ("select_mode", ctypes.c_int32),
                ("max_pairs", ctypes.c_int32)]


class Routing(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_void_p), ("n_shared", ctypes.c_void_p),
                ("shared_mask", ctypes.c_void_p), ("n_res", ctypes.c_void_p),
                ("expert_ids", ctypes.c_void_p), ("weights", ctypes.c_void_p)]


class Stats(ctypes.Structure):
    _fields_ = [("n_valid", ctypes.c_int64), ("hist_b", ctypes.c_int64 * 65),
                ("hist_k", ctypes.c_int64 * 65), ("expert_tokens", ctypes.c_int64 * 65),
                ("activated_blocks", ctypes.c_int64), ("mean_b", ctypes.c_double),
                ("mean_k", ctypes.c_double), ("mean_cb", ctypes.c_double),
                ("activated_gemm_flops", ctypes.c_double), ("routing_flops", ctypes.c_double)]


NORM_MODES = {"none": 0, "pre": 1, "post": 2}


class Block(ctypes.Structure):
    _fields_ = [("norm", ctypes.c_int32), ("residual", ctypes.c_int32),
                ("ln_eps", ctypes.c_float), ("ln_gamma", ctypes.c_void_p),
                ("ln_beta", ctypes.c_void_p), ("b_up", ctypes.c_void_p),
                ("b_down", ctypes.c_void_p)]


EXPORTS = ("unif_moe_route_workspace_size", "unif_moe_route",
           "unif_moe_layer_forward_workspace_size", "unif_moe_layer_forward",
           "unif_moe_layer_forward_profiled", "unif_moe_block_forward_workspace_size",
           "unif_moe_block_forward", "unif_moe_layer_backward_workspace_size",
           "unif_moe_layer_backward", "unif_moe_stats_workspace_size",
           "unif_moe_stats", "unif_moe_layer_forward_static", "unif_moe_forward_work",
           "unif_moe_diversity_loss_workspace_size", "unif_moe_diversity_loss",
           "unif_moe_forward_status", "unif_moe_status_string")
N_PHASE_EVENTS = 7


class Work(ctypes.Structure):
    _fields_ = [("pairs", ctypes.c_int64), ("up_tiles", ctypes.c_int64), ("down_tiles", ctypes.c_int64),
                ("up_mfma_flops", ctypes.c_double), ("down_mfma_flops", ctypes.c_double),
                ("down_parts", ctypes.c_int64), ("down_queued", ctypes.c_int64)]


class UnifMoeError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


_LIB = None


def lib():
    """The loaded HIP library (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing; build it with "
                              "`python -m paper_2608_10392_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, sz = ctypes.c_void_p, ctypes.c_size_t
        cfgp = ctypes.POINTER(Config)
        L.unif_moe_route_workspace_size.argtypes = [cfgp, ctypes.POINTER(sz)]
        L.unif_moe_layer_forward_workspace_size.argtypes = [cfgp, ctypes.POINTER(sz)]
        L.unif_moe_stats_workspace_size.argtypes = [cfgp, ctypes.POINTER(sz)]
        L.unif_moe_route.argtypes = [cfgp, vp, vp, vp, vp, ctypes.POINTER(Routing), vp, sz, vp]
        L.unif_moe_layer_forward.argtypes = [cfgp, vp, vp, vp, vp, vp, vp, vp,
                                             ctypes.POINTER(Routing), vp, sz, vp]
        L.unif_moe_layer_forward_profiled.argtypes = [cfgp, vp, vp, vp, vp, vp, vp, vp,
                                                      ctypes.POINTER(Routing), vp, sz,
                                                      ctypes.POINTER(vp), ctypes.c_int32, vp]
        L.unif_moe_stats.argtypes = [cfgp, ctypes.POINTER(Routing), vp, ctypes.POINTER(Stats),
                                     vp, sz, vp]
        L.unif_moe_layer_backward_workspace_size.argtypes = [cfgp, ctypes.POINTER(sz)]
        L.unif_moe_layer_backward.argtypes = [cfgp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                              vp, sz, vp]
        blkp = ctypes.POINTER(Block)
        L.unif_moe_block_forward_workspace_size.argtypes = [cfgp, blkp, ctypes.POINTER(sz)]
        L.unif_moe_block_forward.argtypes = [cfgp, blkp, vp, vp, vp, vp, vp, vp, vp,
                                             ctypes.POINTER(Routing), vp, sz, vp]
        L.unif_moe_layer_forward_static.argtypes = [cfgp, vp, vp, vp, vp, vp, vp, vp,
                                                    ctypes.POINTER(Routing), vp]
        L.unif_moe_forward_work.argtypes = [cfgp, vp, sz, ctypes.POINTER(Work), vp]
        L.unif_moe_forward_status.argtypes = [cfgp, vp, sz, ctypes.POINTER(ctypes.c_int64), vp]
        L.unif_moe_diversity_loss_workspace_size.argtypes = [cfgp, ctypes.POINTER(sz)]
        L.unif_moe_diversity_loss.argtypes = [cfgp, vp, ctypes.c_float, vp, vp, vp, sz, vp]
        L.unif_moe_status_string.argtypes = [ctypes.c_int32]
        L.unif_moe_status_string.restype = ctypes.c_char_p
        for name in EXPORTS[:-1]:
            getattr(L, name).restype = ctypes.c_int32
        _LIB = L
    return _LIB


def status_string(status):
    return lib().unif_moe_status_string(int(status)).decode()


def make_config(cfg):
    """Config structure from a layer description dict (the keys of
    synth.configs.LAYER_KEYS; modes and dtype as strings)."""
    tau = cfg.get("tau")
    return Config(
        n_tokens=int(cfg["n_tokens"]), d_model=int(cfg["d_model"]),
        n_experts=int(cfg["n_experts"]), n_blocks=int(cfg["n_blocks"]),
        block_width=int(cfg["block_width"]), dtype=DTYPES[cfg["dtype"]],
        tau=math.nan if tau is None else float(tau),
        mass_threshold=float(cfg["mass_threshold"]),
        max_shared=int(cfg["n_blocks"] if cfg.get("max_shared") is None else cfg["max_shared"]),
        alpha_mode=ALPHA_MODES[cfg.get("alpha_mode", "adaptive")],
        alpha_fixed=float(cfg.get("alpha_fixed", 0.0)),
        mass_mode=MASS_MODES[cfg.get("mass_mode", "coupled")],
        fixed_k=int(cfg.get("fixed_k", 1)),
        select_mode=SELECT_MODES[cfg.get("select_mode", "prototype")],
        max_pairs=int(cfg.get("max_pairs", 0) or 0))


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def _check(status, where):
    if status != OK:
        raise UnifMoeError(status, where)


def _size(fn, cfg):
    c = make_config(cfg) if isinstance(cfg, dict) else cfg
    n = ctypes.c_size_t(0)
    _check(getattr(lib(), fn)(ctypes.byref(c), ctypes.byref(n)), fn)
    return n.value


def route_workspace_size(cfg):
    return _size("unif_moe_route_workspace_size", cfg)


def layer_forward_workspace_size(cfg):
    return _size("unif_moe_layer_forward_workspace_size", cfg)


def stats_workspace_size(cfg):
    return _size("unif_moe_stats_workspace_size", cfg)


def _routing_struct(rec):
    if rec is None:
        return None
    return Routing(*(_ptr(rec[k]) for k in ("alpha", "n_shared", "shared_mask", "n_res",
                                            "expert_ids", "weights")))


def alloc_routing(n_tokens, n_experts, device="cuda"):
    """Device arrays of a routing record (torch tensors)."""
    import torch
    N, K = int(n_tokens), int(n_experts)
    return dict(alpha=torch.empty(N, dtype=torch.float32, device=device),
                n_shared=torch.empty(N, dtype=torch.int32, device=device),
                shared_mask=torch.empty(N, dtype=torch.int64, device=device),
                n_res=torch.empty(N, dtype=torch.int32, device=device),
                expert_ids=torch.empty((N, K), dtype=torch.int32, device=device),
                weights=torch.empty((N, K), dtype=torch.float32, device=device))


def alloc_workspace(nbytes, device="cuda"):
    import torch
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def route(cfg, X, valid, W_router, prototypes, out, workspace, stream=None):
    c = make_config(cfg)
    r = _routing_struct(out)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().unif_moe_route(ctypes.byref(c), _ptr(X), _ptr(valid), _ptr(W_router),
                                _ptr(prototypes), ctypes.byref(r), _ptr(workspace), ws_bytes,
                                _stream(stream)), "unif_moe_route")


def layer_forward(cfg, X, valid, W_router, prototypes, W_up, W_down, Y, workspace,
                  routing=None, stream=None):
    c = make_config(cfg)
    r = _routing_struct(routing)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().unif_moe_layer_forward(ctypes.byref(c), _ptr(X), _ptr(valid), _ptr(W_router),
                                        _ptr(prototypes), _ptr(W_up), _ptr(W_down), _ptr(Y),
                                        ctypes.byref(r) if r is not None else None,
                                        _ptr(workspace), ws_bytes, _stream(stream)),
           "unif_moe_layer_forward")


STATIC_WORKSPACE_BYTES = 128 << 20   # UNIF_MOE_STATIC_WORKSPACE_BYTES


def layer_forward_static(cfg, X, valid, W_router, prototypes, W_up, W_down, Y, routing=None,
                         stream=None):
    """layer_forward with the library's static per-GPU scratch instead of a
    caller workspace (unif_moe_layer_forward_static)."""
    c = make_config(cfg)
    r = _routing_struct(routing)
    _check(lib().unif_moe_layer_forward_static(ctypes.byref(c), _ptr(X), _ptr(valid), _ptr(W_router),
                                               _ptr(prototypes), _ptr(W_up), _ptr(W_down), _ptr(Y),
                                               ctypes.byref(r) if r is not None else None,
                                               _stream(stream)),
           "unif_moe_layer_forward_static")


def layer_forward_profiled(cfg, X, valid, W_router, prototypes, W_up, W_down, Y, workspace,
                           events, routing=None, stream=None):
    """As layer_forward, recording the seven torch.cuda.Event objects in
    ``events`` at the phase boundaries (see the C header)."""
    c = make_config(cfg)
    r = _routing_struct(routing)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    handles = (ctypes.c_void_p * N_PHASE_EVENTS)(*(ev.cuda_event for ev in events))
    _check(lib().unif_moe_layer_forward_profiled(
        ctypes.byref(c), _ptr(X), _ptr(valid), _ptr(W_router), _ptr(prototypes), _ptr(W_up),
        _ptr(W_down), _ptr(Y), ctypes.byref(r) if r is not None else None, _ptr(workspace),
        ws_bytes, handles, N_PHASE_EVENTS, _stream(stream)), "unif_moe_layer_forward_profiled")


def make_block(blk):
    """Block structure from a dict: norm ("none", "pre", "post"), residual,
    ln_eps, and device tensors (or None) ln_gamma, ln_beta, b_up, b_down."""
    return Block(norm=NORM_MODES[blk["norm"]], residual=1 if blk["residual"] else 0,
                 ln_eps=float(blk["ln_eps"]), ln_gamma=_ptr(blk.get("ln_gamma")),
                 ln_beta=_ptr(blk.get("ln_beta")), b_up=_ptr(blk.get("b_up")),
                 b_down=_ptr(blk.get("b_down")))


def block_forward_workspace_size(cfg, blk):
    c = make_config(cfg) if isinstance(cfg, dict) else cfg
    b = make_block(blk) if isinstance(blk, dict) else blk
    n = ctypes.c_size_t(0)
    _check(lib().unif_moe_block_forward_workspace_size(ctypes.byref(c), ctypes.byref(b),
                                                       ctypes.byref(n)),
           "unif_moe_block_forward_workspace_size")
    return n.value


def block_forward(cfg, blk, X, valid, W_router, prototypes, W_up, W_down, Y, workspace,
                  routing=None, stream=None):
    c = make_config(cfg)
    b = make_block(blk)
    r = _routing_struct(routing)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().unif_moe_block_forward(ctypes.byref(c), ctypes.byref(b), _ptr(X), _ptr(valid),
                                        _ptr(W_router), _ptr(prototypes), _ptr(W_up),
                                        _ptr(W_down), _ptr(Y),
                                        ctypes.byref(r) if r is not None else None,
                                        _ptr(workspace), ws_bytes, _stream(stream)),
           "unif_moe_block_forward")


def layer_backward_workspace_size(cfg):
    return _size("unif_moe_layer_backward_workspace_size", cfg)


def layer_backward(cfg, X, valid, W_router, prototypes, W_up, W_down, dY, dX, dW_up, dW_down,
                   dW_router, workspace, stream=None):
    c = make_config(cfg)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().unif_moe_layer_backward(ctypes.byref(c), _ptr(X), _ptr(valid), _ptr(W_router),
                                         _ptr(prototypes), _ptr(W_up), _ptr(W_down), _ptr(dY),
                                         _ptr(dX), _ptr(dW_up), _ptr(dW_down), _ptr(dW_router),
                                         _ptr(workspace), ws_bytes, _stream(stream)),
           "unif_moe_layer_backward")


def diversity_loss_workspace_size(cfg):
    return _size("unif_moe_diversity_loss_workspace_size", cfg)


def diversity_loss(cfg, W_router, lam, loss, dW_router, workspace, stream=None):
    """L_div into ``loss`` (1 fp32) and dW_router += lam * dL_div/dW_router."""
    c = make_config(cfg)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().unif_moe_diversity_loss(ctypes.byref(c), _ptr(W_router), float(lam), _ptr(loss),
                                         _ptr(dW_router), _ptr(workspace), ws_bytes, _stream(stream)),
           "unif_moe_diversity_loss")


def stats(cfg, routing, valid, workspace, stream=None):
    c = make_config(cfg)
    r = _routing_struct(routing)
    s = Stats()
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().unif_moe_stats(ctypes.byref(c), ctypes.byref(r), _ptr(valid), ctypes.byref(s),
                                _ptr(workspace), ws_bytes, _stream(stream)), "unif_moe_stats")
    return dict(n_valid=s.n_valid, hist_b=list(s.hist_b), hist_k=list(s.hist_k),
                expert_tokens=list(s.expert_tokens), activated_blocks=s.activated_blocks,
                mean_b=s.mean_b, mean_k=s.mean_k, mean_cb=s.mean_cb,
                activated_gemm_flops=s.activated_gemm_flops, routing_flops=s.routing_flops)


def forward_work(cfg, workspace, stream=None):
    """Work the last forward in ``workspace`` executed (unif_moe_forward_work)."""
    c = make_config(cfg)
    w = Work()
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().unif_moe_forward_work(ctypes.byref(c), _ptr(workspace), ws_bytes, ctypes.byref(w),
                                       _stream(stream)), "unif_moe_forward_work")
    return dict(pairs=w.pairs, up_tiles=w.up_tiles, down_tiles=w.down_tiles,
                up_mfma_flops=w.up_mfma_flops, down_mfma_flops=w.down_mfma_flops,
                down_parts=w.down_parts, down_queued=w.down_queued)



def forward_status(cfg, workspace, stream=None):
    """(status, pairs) of the last forward in ``workspace``
    (unif_moe_forward_status): status is OK or ECAPACITY (the routing needed
    more pairs than cfg's max_pairs); other codes raise."""
    c = make_config(cfg)
    n = ctypes.c_int64(0)
    ws_bytes = workspace.numel() * workspace.element_size()
    s = lib().unif_moe_forward_status(ctypes.byref(c), _ptr(workspace), ws_bytes, ctypes.byref(n),
                                      _stream(stream))
    if s not in (OK, ECAPACITY):
        _check(s, "unif_moe_forward_status")
    return s, n.value
