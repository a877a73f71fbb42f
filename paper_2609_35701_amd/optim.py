"""MeqMuon over torch parameters (Algorithm "MeqMuon", arxiv 2609.35701, Section "MeqMuon").

Argument marshalling only: each parameter kind runs through libmeq's C ABI and HIP kernels
(``meq_init_kind`` / ``meq_step``).  The three branches of the algorithm:
  hidden   2D hidden-layer weights: Newton-Schulz + adaptive one-sided normalization (eq. "hidden")
  aux      remaining 2D parameters (token embeddings, LM head): two-sided normalization (eq. "aux")
  vectors  1-D parameters (norm weights, biases): global-RMS normalization (eq. "vector")
all with the momentum of eq. "momentum" and the write-back of eq. "meqmuon-update".
"""
from __future__ import annotations

from typing import Dict, Iterable, List, Optional, Tuple

import torch

from . import meq


def split_parameters(model) -> Tuple[list, list, list]:
    """(hidden, aux, vectors) parameters of a torch module.

    aux: the weights of ``nn.Embedding`` modules and of a module named ``lm_head`` (tied weights
    are listed once).  vectors: every parameter with one dimension.  hidden: the other 2D
    parameters.  Parameters with more than two dimensions are rejected: the update is defined
    for matrices and vectors."""
    aux_ids = set()
    for name, mod in model.named_modules():
        if isinstance(mod, torch.nn.Embedding) or name.split(".")[-1] == "lm_head":
            w = getattr(mod, "weight", None)
            if w is not None:
                aux_ids.add(id(w))
    hidden, aux, vectors, seen = [], [], [], set()
    for name, p in model.named_parameters():
        if id(p) in seen or not p.requires_grad:
            continue
        seen.add(id(p))
        if p.dim() == 1:
            vectors.append(p)
        elif p.dim() == 2:
            (aux if id(p) in aux_ids else hidden).append(p)
        else:
            raise ValueError(f"parameter {name} has {p.dim()} dimensions; MeqMuon takes matrices and vectors")
    return hidden, aux, vectors


class MeqMuon(torch.optim.Optimizer):
    """One optimizer over the three parameter kinds, with the ``torch.optim.Optimizer`` interface.

    Each kind is one parameter group (``group["kind"]`` is ``meq.PARAM_HIDDEN``, ``PARAM_AUX`` or
    ``PARAM_VECTOR``) whose ``lr`` is read at every step, so the learning-rate schedulers of
    ``torch.optim.lr_scheduler`` drive it.  Parameters of one kind may mix bf16 and fp32; each
    (kind, dtype) pair gets its own plan, momenta and workspace.  ``step()`` reads ``p.grad`` of
    every parameter (same dtype and shape as the parameter) and enqueues all updates on the
    current torch stream.  ``hidden_hparams`` overrides the hyperparameters of the hidden weights
    only (for instance Nesterov momentum, as in the paper's experiments, or the Moonlight-Muon
    rule)."""

    def __init__(self, hidden: Iterable = (), aux: Iterable = (), vectors: Iterable = (), lr: float = 0.02,
                 hparams: Optional[meq.HParams] = None, hidden_hparams: Optional[meq.HParams] = None):
        kinds = [(meq.PARAM_HIDDEN, list(hidden)), (meq.PARAM_AUX, list(aux)), (meq.PARAM_VECTOR, list(vectors))]
        super().__init__([{"params": ps, "kind": kind} for kind, ps in kinds if ps], {"lr": float(lr)})
        base = hparams if hparams is not None else meq.default_hparams()
        # (parameter group, plan) pairs, one plan per (kind, dtype)
        self.updates: List[Tuple[int, meq.ParamUpdate]] = []
        self._group_of: List[int] = []
        for gi, group in enumerate(self.param_groups):
            kind = group["kind"]
            hp = (hidden_hparams or base) if kind == meq.PARAM_HIDDEN else base
            by_dtype: Dict[object, list] = {}
            for p in group["params"]:
                by_dtype.setdefault(p.dtype, []).append(p)
            for _, ps in sorted(by_dtype.items(), key=lambda kv: str(kv[0])):
                self.updates.append((kind, meq.ParamUpdate(ps, hp, kind=kind)))
                self._group_of.append(gi)

    @classmethod
    def for_model(cls, model, **kw) -> "MeqMuon":
        hidden, aux, vectors = split_parameters(model)
        return cls(hidden, aux, vectors, **kw)

    @torch.no_grad()
    def step(self, closure=None, lr: Optional[float] = None):
        """One update of every parameter.  ``lr`` overrides the groups' learning rates for this
        step only; ``closure`` (re-evaluating the loss) is called first, as in torch optimizers."""
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        for gi, (_, upd) in zip(self._group_of, self.updates):
            step_lr = float(lr) if lr is not None else float(self.param_groups[gi]["lr"])
            grads = []
            for p in upd.params:
                if p.grad is None:
                    raise ValueError("every parameter needs a gradient (p.grad) for a MeqMuon step")
                grads.append(p.grad if p.grad.is_contiguous() else p.grad.contiguous())
            upd.step(grads, step_lr)
        return loss

    def state_dict(self) -> dict:
        """torch's optimizer state (the parameter groups and their learning rates) plus the fp32
        momenta, one list per plan in construction order."""
        state = super().state_dict()
        state["momenta"] = [[b.detach().clone() for b in upd.momenta] for _, upd in self.updates]
        return state

    def load_state_dict(self, state: dict) -> None:
        moms = state["momenta"]
        if len(moms) != len(self.updates) or any(len(ms) != len(upd.momenta) for (_, upd), ms in zip(self.updates, moms)):
            raise ValueError("state does not match this optimizer's plans")
        super().load_state_dict({k: v for k, v in state.items() if k != "momenta"})
        with torch.no_grad():
            for (_, upd), ms in zip(self.updates, moms):
                for b, m in zip(upd.momenta, ms):
                    b.copy_(m)
