"""Device-resident UniF-MoE layer: moves one layer's inputs to the GPU once
and calls the HIP library on them (torch supplies memory and streams)."""
import numpy as np

from . import _lib


def to_device(a, dtype_name, device):
    """numpy array -> torch device tensor; bf16 data arrives as uint16 bits."""
    import torch
    if a is None:
        return None
    if dtype_name == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device)


class DeviceLayer:
    """Inputs of one layer on the device, plus output, record and workspace.

    ``cfg`` is a layer description dict (dtype "bf16" or "f32"); arrays are
    numpy: X and the expert weights as bf16 bits (uint16) or float32, the
    router and prototypes as float32, ``valid`` as uint8 or None.
    """

    def __init__(self, cfg, X, valid, W_router, prototypes, W_up=None, W_down=None,
                 device="cuda:0"):
        import torch
        self.cfg = dict(cfg)
        self.device = device
        dt = cfg["dtype"]
        N, d, K = cfg["n_tokens"], cfg["d_model"], cfg["n_experts"]
        self.X = to_device(X, dt, device)
        self.valid = None if valid is None else torch.from_numpy(np.ascontiguousarray(valid, np.uint8)).to(device)
        self.W_router = to_device(np.asarray(W_router, np.float32), "f32", device)
        self.prototypes = to_device(np.asarray(prototypes, np.float32), "f32", device)
        self.W_up = to_device(W_up, dt, device)
        self.W_down = to_device(W_down, dt, device)
        self.Y = torch.empty((N, d), dtype=torch.bfloat16 if dt == "bf16" else torch.float32,
                             device=device)
        self.routing = _lib.alloc_routing(N, K, device)
        self.ws_forward = None
        self.ws_route = None
        self.ws_stats = None

    def forward(self, stream=None, routing=True):
        if self.ws_forward is None:
            self.ws_forward = _lib.alloc_workspace(_lib.layer_forward_workspace_size(self.cfg), self.device)
        _lib.layer_forward(self.cfg, self.X, self.valid, self.W_router, self.prototypes,
                           self.W_up, self.W_down, self.Y, self.ws_forward,
                           routing=self.routing if routing else None, stream=stream)
        return self.Y

    def block_forward(self, blk, X=None, stream=None, routing=True):
        """The transformer block around the layer (``blk`` as
        synth.block_inputs returns it: numpy parameters, moved to the device
        on each call). ``X`` replaces the layer input (the residual stream)."""
        dt = self.cfg["dtype"]
        Xd = self.X if X is None else to_device(X, dt, self.device)
        b = dict(norm=blk["norm"], residual=blk["residual"], ln_eps=blk["ln_eps"])
        for k in ("ln_gamma", "ln_beta", "b_up", "b_down"):
            b[k] = None if blk.get(k) is None else to_device(np.asarray(blk[k], np.float32), "f32",
                                                              self.device)
        ws = _lib.alloc_workspace(_lib.block_forward_workspace_size(self.cfg, b), self.device)
        _lib.block_forward(self.cfg, b, Xd, self.valid, self.W_router, self.prototypes,
                           self.W_up, self.W_down, self.Y, ws,
                           routing=self.routing if routing else None, stream=stream)
        return self.Y

    def backward(self, dY, stream=None):
        """Gradients of sum(dY * Y) (numpy dY in the layer's format): dict of
        fp32 device tensors dX, dW_up, dW_down, dW_router."""
        import torch
        c = self.cfg
        N, d, K = c["n_tokens"], c["d_model"], c["n_experts"]
        H = c["n_blocks"] * c["block_width"]
        f = dict(dtype=torch.float32, device=self.device)
        g = dict(dX=torch.empty((N, d), **f), dW_up=torch.empty((K + 1, H, d), **f),
                 dW_down=torch.empty((K + 1, d, H), **f), dW_router=torch.empty((K + 1, d), **f))
        dYd = to_device(dY, c["dtype"], self.device)
        ws = _lib.alloc_workspace(_lib.layer_backward_workspace_size(c), self.device)
        _lib.layer_backward(c, self.X, self.valid, self.W_router, self.prototypes, self.W_up,
                            self.W_down, dYd, g["dX"], g["dW_up"], g["dW_down"], g["dW_router"], ws,
                            stream=stream)
        return g

    def route(self, out=None, stream=None):
        if self.ws_route is None:
            self.ws_route = _lib.alloc_workspace(_lib.route_workspace_size(self.cfg), self.device)
        out = self.routing if out is None else out
        _lib.route(self.cfg, self.X, self.valid, self.W_router, self.prototypes, out,
                   self.ws_route, stream=stream)
        return out

    def stats(self, stream=None):
        if self.ws_stats is None:
            self.ws_stats = _lib.alloc_workspace(_lib.stats_workspace_size(self.cfg), self.device)
        return _lib.stats(self.cfg, self.routing, self.valid, self.ws_stats, stream=stream)

    def routing_numpy(self):
        r = {k: v.cpu().numpy() for k, v in self.routing.items()}
        r["shared_mask"] = r["shared_mask"].view(np.uint64)
        return r

    def output_numpy(self):
        import torch
        if self.cfg["dtype"] == "bf16":
            return self.Y.view(torch.int16).cpu().numpy().view(np.uint16)
        return self.Y.cpu().numpy()
