"""M-FAC preconditioned SGD on a PyTorch model (Section 4.2, Application 2).

Each step inserts the new gradient g_t into a sliding window of the last m
gradients (replacing the oldest) and moves the weights along the
preconditioned direction:

    w <- w - lr * F^-1 g_t,   F = damp * I + (1/m) sum_{tau < m} g_{t-tau} g_{t-tau}^T

(the damping is the lambda * I of eq. 2's base case, as everywhere in this
package). No momentum, as in the paper's optimizer experiments. Weight decay,
when set, is added to the gradient before it enters the window (w's decay is
preconditioned together with the loss gradient).

The window insert and F^-1 g_t are one `mfac_window_replace` call (two passes
over the window in the library's kernels). Gathering the parameter gradients
into one flat vector and applying the update are multi-tensor copies/axpys
on views of two flat buffers. Until m steps have run, the empty slots are
zero rows and the 1/m scale stays that of the full window (Theorem 1 with a
partially filled sum).
"""

import torch

from ._binding import Window


class MFAC(torch.optim.Optimizer):
    """M-FAC optimizer over all parameters of the given groups (fp32, one GPU).

    Args:
        params: iterable of parameters or parameter groups (all float32, on one
            CUDA device, dense gradients).
        lr: learning rate (per group).
        m: window size (number of gradients kept).
        damp: damping lambda of F = lambda I + G^T G / m.
        weight_decay: coupled L2 decay added to the gradient (per group).
    """

    def __init__(self, params, lr, m=512, damp=1e-4, weight_decay=0.0):
        if lr <= 0 or m < 1 or damp <= 0 or weight_decay < 0:
            raise ValueError("MFAC: need lr > 0, m >= 1, damp > 0, weight_decay >= 0")
        super().__init__(params, dict(lr=lr, weight_decay=weight_decay))
        plist = [p for g in self.param_groups for p in g["params"]]
        if not plist:
            raise ValueError("MFAC: no parameters")
        dev = plist[0].device
        for p in plist:
            if p.device != dev or p.device.type != "cuda" or p.dtype != torch.float32:
                raise ValueError("MFAC: all parameters must be float32 on one CUDA device")
        self.m, self.damp = int(m), float(damp)
        self.d = sum(p.numel() for p in plist)
        self.device = dev
        with torch.cuda.device(dev):
            self.window = Window(self.d, self.m, self.damp, device=dev)
        self._g = torch.zeros(self.d, dtype=torch.float32, device=dev)
        self._y = torch.zeros(self.d, dtype=torch.float32, device=dev)
        # per-group views of the flat gradient and update vectors, in parameter order
        self._views = []
        off = 0
        for group in self.param_groups:
            gv, yv = [], []
            for p in group["params"]:
                n = p.numel()
                gv.append(self._g[off:off + n].view_as(p))
                yv.append(self._y[off:off + n].view_as(p))
                off += n
            self._views.append((gv, yv))
        self.steps = 0

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        for group, (gv, _) in zip(self.param_groups, self._views):
            ps = group["params"]
            grads = [p.grad if p.grad is not None else torch.zeros_like(p) for p in ps]
            for p, g in zip(ps, grads):
                if g.is_sparse:
                    raise RuntimeError("MFAC: sparse gradients are not supported")
            torch._foreach_copy_(gv, grads)
            if group["weight_decay"]:
                torch._foreach_add_(gv, ps, alpha=group["weight_decay"])
        # the library enqueues on the window's stream: follow the stream this
        # step runs on, so the copies into _g above and the update below are
        # ordered with the window's passes
        cur = torch.cuda.current_stream(self.device).cuda_stream
        if cur != self.window.stream:
            self.window.set_stream()
        self.window.replace(self._g, y_out=self._y)
        for group, (_, yv) in zip(self.param_groups, self._views):
            torch._foreach_add_(group["params"], yv, alpha=-group["lr"])
        self.steps += 1
        return loss

    def preconditioned(self):
        """F^-1 g of the last step (a view of the flat update vector)."""
        return self._y

    def status(self):
        """Library status of the window (0 = ok; a device-side error is latched
        and returned once)."""
        return self.window.status()

    def state_dict(self):
        sd = super().state_dict()
        head, steps = self.window.info()
        sd["mfac"] = {"rows": self.window.get_rows().cpu(), "head": head, "window_steps": steps,
                      "steps": self.steps, "m": self.m, "damp": self.damp, "d": self.d}
        return sd

    def load_state_dict(self, state_dict):
        st = dict(state_dict)
        mf = st.pop("mfac", None)
        super().load_state_dict(st)
        if mf is not None:
            if (mf["m"], mf["d"]) != (self.m, self.d) or mf["damp"] != self.damp:
                raise ValueError("MFAC: window shape or damping differs from the checkpoint")
            self.window.set_rows(0, mf["rows"].to(self.device).contiguous())
            self.window.rebuild()
            self.window.set_head(mf["head"], mf["window_steps"])
            self.steps = mf["steps"]
