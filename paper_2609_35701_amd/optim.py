"""MeqMuon over torch parameters (Algorithm "MeqMuon", arxiv 2609.35701, Section "MeqMuon").

Argument marshalling only: each parameter kind runs through libmeq's C ABI and HIP kernels
(``meq_init_kind`` / ``meq_step``).  The three branches of the algorithm:
  hidden   2D hidden-layer weights: Newton-Schulz + adaptive one-sided normalization (eq. "hidden")
  aux      remaining 2D parameters (token embeddings, LM head): two-sided normalization (eq. "aux")
  vectors  1-D parameters (norm weights, biases): global-RMS normalization (eq. "vector")
all with the momentum of eq. "momentum" and the write-back of eq. "meqmuon-update".
"""
from __future__ import annotations

from typing import Dict, Iterable, List, Optional, Sequence, Tuple

from . import meq


def split_parameters(model) -> Tuple[list, list, list]:
    """(hidden, aux, vectors) parameters of a torch module.

    aux: the weights of ``nn.Embedding`` modules and of a module named ``lm_head`` (tied weights
    are listed once).  vectors: every parameter with one dimension.  hidden: the other 2D
    parameters.  Parameters with more than two dimensions are rejected: the update is defined
    for matrices and vectors."""
    import torch

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


class MeqMuon:
    """One optimizer over the three parameter kinds.

    Parameters of one kind may mix bf16 and fp32; each (kind, dtype) pair gets its own plan,
    momenta and workspace.  ``step(lr)`` reads ``p.grad`` of every parameter (same dtype and shape
    as the parameter) and enqueues all updates on the current torch stream.  ``hidden_hparams``
    overrides the hyperparameters of the hidden weights only (for instance Nesterov momentum, as
    in the paper's experiments, or the Moonlight-Muon rule)."""

    def __init__(self, hidden: Iterable = (), aux: Iterable = (), vectors: Iterable = (), lr: float = 0.02,
                 hparams: Optional[meq.HParams] = None, hidden_hparams: Optional[meq.HParams] = None):
        self.lr = float(lr)
        base = hparams if hparams is not None else meq.default_hparams()
        self.updates: List[Tuple[int, meq.ParamUpdate]] = []
        for kind, params, hp in ((meq.PARAM_HIDDEN, hidden, hidden_hparams or base),
                                 (meq.PARAM_AUX, aux, base), (meq.PARAM_VECTOR, vectors, base)):
            by_dtype: Dict[object, list] = {}
            for p in params:
                by_dtype.setdefault(p.dtype, []).append(p)
            for _, ps in sorted(by_dtype.items(), key=lambda kv: str(kv[0])):
                self.updates.append((kind, meq.ParamUpdate(ps, hp, kind=kind)))

    @classmethod
    def for_model(cls, model, **kw) -> "MeqMuon":
        hidden, aux, vectors = split_parameters(model)
        return cls(hidden, aux, vectors, **kw)

    def step(self, lr: Optional[float] = None) -> None:
        lr = self.lr if lr is None else float(lr)
        for _, upd in self.updates:
            grads = []
            for p in upd.params:
                if p.grad is None:
                    raise ValueError("every parameter needs a gradient (p.grad) for a MeqMuon step")
                grads.append(p.grad if p.grad.is_contiguous() else p.grad.contiguous())
            upd.step(grads, lr)

    def zero_grad(self) -> None:
        for _, upd in self.updates:
            for p in upd.params:
                p.grad = None

    def state_dict(self) -> dict:
        """Momenta (fp32, one per parameter, in construction order per plan) and the learning rate."""
        return {"lr": self.lr, "momenta": [[b.detach().clone() for b in upd.momenta] for _, upd in self.updates]}

    def load_state_dict(self, state: dict) -> None:
        moms = state["momenta"]
        if len(moms) != len(self.updates):
            raise ValueError("state does not match this optimizer's plans")
        for (_, upd), ms in zip(self.updates, moms):
            if len(ms) != len(upd.momenta):
                raise ValueError("state does not match this optimizer's plans")
            for b, m in zip(upd.momenta, ms):
                b.copy_(m)
        self.lr = float(state.get("lr", self.lr))
