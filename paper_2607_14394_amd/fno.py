"""FNO forward on the shards of a decomposed (x, y, z, t) grid, run one after
another on one GPU: the lift P, L Fourier layers (each as Algorithm 1: the
forward partial DFT of every shard summed into one spectrum, the mode-wise
channel mix over the mode ranges S_p, then per shard the inverse partial DFT,
the point-wise bypass and GELU), and the projection Q (Sec. II).

Orchestration only: every step is a call of the DTST library
(``dtst_pointwise``, ``dtst_forward``, ``dtst_mix``, ``dtst_inverse_block``);
no arithmetic happens here.  P and Q are single linear layers with a bias and
every Fourier layer, the last included, ends in GELU (Algorithm 1).
"""

from __future__ import annotations

from . import Plan, dtst_pointwise


class FNO:
    """descs: one spectral-layer descriptor per shard (same global grid,
    modes and batch; c_in = c_out = d_v).  lift = (w (d_v, C_in), b (d_v,)),
    layers = [(R (M, d_v, d_v) complex64, W (d_v, d_v) float32), ...],
    proj = (w (C_out, d_v), b (C_out,)); all device tensors, used as given.
    flags: plan flags of every shard's plan (PLAN_UNFUSED_BLOCK runs each
    block epilogue as the inverse followed by the separate epilogue)."""

    def __init__(self, descs, lift, layers, proj, device="cuda", flags=0):
        import torch
        self.plans = [Plan(d, device, flags) for d in descs]
        p0 = self.plans[0]
        d = p0.desc
        self.dv = d.c_in
        if d.c_out != self.dv:
            raise ValueError("the Fourier layers map d_v channels to d_v channels (c_in = c_out)")
        for p in self.plans[1:]:
            q = p.desc
            if (tuple(q.n_global) != tuple(d.n_global) or tuple(q.kmax) != tuple(d.kmax) or q.kt != d.kt
                    or q.batch != d.batch or q.c_in != d.c_in or q.c_out != d.c_out):
                raise ValueError("every shard needs the same global grid, modes, batch and channels")
        self.lift, self.layers, self.proj = lift, list(layers), proj
        self.c_in, self.c_out = lift[0].shape[1], proj[0].shape[0]
        if tuple(lift[0].shape) != (self.dv, self.c_in) or tuple(proj[0].shape) != (self.c_out, self.dv):
            raise ValueError("lift w must be (d_v, C_in) and proj w (C_out, d_v)")
        M = p0.n_modes
        for r, w in self.layers:
            if tuple(r.shape) != (M, self.dv, self.dv) or tuple(w.shape) != (self.dv, self.dv):
                raise ValueError(f"each layer needs R ({M}, {self.dv}, {self.dv}) and W ({self.dv}, {self.dv})")
        P = len(self.plans)
        self.ranges = [((M * r) // P, (M * (r + 1)) // P) for r in range(P)]
        f32 = torch.float32
        self.va = [torch.empty(p.spatial_shape(self.dv), dtype=f32, device=device) for p in self.plans]
        self.vb = [torch.empty(p.spatial_shape(self.dv), dtype=f32, device=device) for p in self.plans]
        self.xhat = torch.empty(p0.spectral_shape(self.dv), dtype=torch.complex64, device=device)
        self.yhat = torch.empty_like(self.xhat)

    def input_shape(self, shard):
        return self.plans[shard].spatial_shape(self.c_in)

    def output_shape(self, shard):
        return self.plans[shard].spatial_shape(self.c_out)

    def forward(self, xs, outs, stream=None):
        """xs[p]: (B, C_in, shard p) float32, outs[p]: (B, C_out, shard p)."""
        va, vb = self.va, self.vb
        for x, v in zip(xs, va):
            dtst_pointwise(x, self.lift[0], self.lift[1], v, act=0, stream=stream)
        for r, w in self.layers:
            for p, (plan, v) in enumerate(zip(self.plans, va)):
                plan.forward(v, self.xhat, accumulate=p > 0, stream=stream)
            for m0, m1 in self.ranges:
                self.plans[0].mix(self.xhat, r[m0:m1], self.yhat, m0, m1, stream=stream)
            for plan, v, u in zip(self.plans, va, vb):
                plan.inverse_block(self.yhat, v, w, u, stream=stream)
            va, vb = vb, va
        for v, y in zip(va, outs):
            dtst_pointwise(v, self.proj[0], self.proj[1], y, act=0, stream=stream)

    def close(self):
        for p in self.plans:
            p.close()
