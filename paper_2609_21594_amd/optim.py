"""A torch optimizer over the library: Muon for the matrix parameters and a
chained AdamW for the others (Sec. 6.4 hands the one-dimensional and scalar
parameters to AdamW through a chained optimizer).

Each `step()` makes one `muon_step` call per parameter group over all of the
group's matrix parameters (2-D, or [E, M, N] stacks of independent matrices,
Sec. 6.3) and one `muon_adamw_step` call per group and step count over the
rest (a parameter whose first gradient comes late has its own count).  The
state
lives in torch tensors (`momentum_buffer`; `exp_avg`, `exp_avg_sq`, `step`),
so `state_dict()` and `load_state_dict()` checkpoint and restore it.  Python
only gathers arguments; every update runs in the library's kernels.
"""
from __future__ import annotations

import torch

from .binding import Muon


def _is_matrix(p: torch.Tensor, group) -> bool:
    use = group.get("use_muon")
    if use is not None:
        return bool(use)
    return p.dim() in (2, 3)


class MuonAdamW(torch.optim.Optimizer):
    """Muon (momentum, Newton-Schulz orthogonalisation, RMS-matched scale,
    decoupled decay) for matrix parameters, AdamW for the others.

    Per group: `lr`, `momentum` (beta), `nesterov`, `weight_decay`,
    `ns_steps`, `ns_coeffs` (a K x 3 table or None for the constant quintic),
    `ns_precision` ("bf16" or "f32"), `scale_mode` (0: 0.2 sqrt(max(m, n)),
    1: none, 2: sqrt(max(1, m/n))), `eps`; and for the AdamW part
    `adamw_lr`, `adamw_betas`, `adamw_eps`, `adamw_weight_decay`.  A group
    may set `use_muon` to force its parameters to one side.  Parameters are
    bf16 or fp32 tensors on one GPU with contiguous columns; gradients have
    the parameter's layout."""

    def __init__(self, params, lr=0.02, momentum=0.95, nesterov=True, weight_decay=0.0, ns_steps=5,
                 ns_coeffs=None, ns_precision="bf16", scale_mode=0, eps=1e-7, adamw_lr=3e-4,
                 adamw_betas=(0.9, 0.95), adamw_eps=1e-8, adamw_weight_decay=0.0):
        defaults = dict(lr=lr, momentum=momentum, nesterov=nesterov, weight_decay=weight_decay,
                        ns_steps=ns_steps, ns_coeffs=ns_coeffs, ns_precision=ns_precision,
                        scale_mode=scale_mode, eps=eps, adamw_lr=adamw_lr, adamw_betas=adamw_betas,
                        adamw_eps=adamw_eps, adamw_weight_decay=adamw_weight_decay)
        super().__init__(params, defaults)
        devices = {p.device for g in self.param_groups for p in g["params"]}
        if len(devices) != 1 or next(iter(devices)).type != "cuda":
            raise ValueError("MuonAdamW needs every parameter on one GPU")
        self._device = next(iter(devices)).index or 0
        self._lib = Muon(self._device)

    def load_state_dict(self, state_dict):
        """As torch's, except that the moments stay fp32: torch casts floating
        state to each parameter's dtype, which for bf16 parameters would
        round the momentum and AdamW moments.  The saved tensors are copied
        back exactly."""
        super().load_state_dict(state_dict)
        by_id = {pid: p for saved, g in zip(state_dict["param_groups"], self.param_groups)
                 for pid, p in zip(saved["params"], g["params"])}
        for pid, st in state_dict["state"].items():
            p = by_id[pid]
            for k, v in st.items():
                if k != "step" and torch.is_tensor(v):
                    self.state[p][k] = v.to(device=p.device, dtype=torch.float32, copy=True)

    def close(self):
        """Releases the library handle (its workspace)."""
        if getattr(self, "_lib", None) is not None:
            self._lib.close()
            self._lib = None

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        for group in self.param_groups:
            mats, mgrads, moms = [], [], []
            vecs, vgrads, ms, vs, steps = [], [], [], [], []
            for p in group["params"]:
                if p.grad is None:
                    continue
                if p.grad.is_sparse:
                    raise RuntimeError("MuonAdamW does not take sparse gradients")
                st = self.state[p]
                if _is_matrix(p, group):
                    if "momentum_buffer" not in st:
                        st["momentum_buffer"] = torch.zeros(p.shape, dtype=torch.float32, device=p.device)
                    mats.append(p)
                    mgrads.append(p.grad)
                    moms.append(st["momentum_buffer"])
                else:
                    if "step" not in st:
                        st["step"] = torch.zeros((), dtype=torch.int64)
                        st["exp_avg"] = torch.zeros(p.shape, dtype=torch.float32, device=p.device)
                        st["exp_avg_sq"] = torch.zeros(p.shape, dtype=torch.float32, device=p.device)
                    st["step"] += 1
                    vecs.append(p)
                    vgrads.append(p.grad)
                    ms.append(st["exp_avg"])
                    vs.append(st["exp_avg_sq"])
                    steps.append(int(st["step"]))
            if mats:
                self._lib.step(mats, mgrads, moms, lr=group["lr"], beta=group["momentum"],
                               weight_decay=group["weight_decay"], eps=group["eps"],
                               ns_steps=group["ns_steps"], nesterov=group["nesterov"],
                               ns_coeffs=group["ns_coeffs"], ns_precision=group["ns_precision"],
                               scale_mode=group["scale_mode"])
            # one call per distinct step count (parameters that joined later
            # have their own bias correction)
            for t in sorted(set(steps)):
                idx = [i for i, s in enumerate(steps) if s == t]
                self._lib.adamw_step([vecs[i] for i in idx], [vgrads[i] for i in idx],
                                     [ms[i] for i in idx], [vs[i] for i in idx], t,
                                     lr=group["adamw_lr"], betas=tuple(group["adamw_betas"]),
                                     eps=group["adamw_eps"], weight_decay=group["adamw_weight_decay"])
        return loss
