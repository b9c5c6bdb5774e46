"""Prune policies on the library's kernels.

Lethe and the baselines the paper compares against differ only in the
parameters they hand to the same calls; every budget, selection and
compaction still runs in liblethe's kernels:

* ``lethe``: decayed scores (Eq. 5, gamma < 1), layer budgets from each
  layer's Hoyer sparsity (Eq. 1 on Eq. 2's head sum), RASR selection per KV
  head with a recent window (RASR section).
* ``lethe-shared``: the same, with one kept set per (layer, sequence) ranked
  by the head-summed score (Eq. 2 read literally).
* ``h2o``: heavy hitters by cumulative attention (gamma = 1) plus a recent
  window, the same budget in every layer.
* ``streaming``: attention sinks plus a recent window (StreamingLLM); the
  window grows to fill the budget, scores are not consulted.
* ``pyramid``: PyramidKV's static layer budgets, falling linearly with depth
  (first : last = 2 beta - 1), RASR selection per KV head.  Every layer first
  keeps its protected rows (recent + sink, the split's floors); the
  progression shapes the budget above them.

Uniform and pyramid budgets go through lethe_layer_sparsity's ``sparsity_in``
argument: the split gives layer l a share proportional to
1 + floor((1 - S_l) 2^24), so S_l = 1 - w_l / max(w) turns a static weight
table into the same integer split (sum exactly the global budget, floors and
caps honoured).
"""
import math
from dataclasses import dataclass

from . import lethe as L

POLICY_NAMES = ("lethe", "lethe-shared", "h2o", "streaming", "pyramid")


@dataclass(frozen=True)
class Policy:
    name: str
    gamma: float
    sink: int
    layer_budget: str      # "sparsity", "uniform", "pyramid"
    shared: bool = False   # one kept set per (layer, sequence)
    window_fills: bool = False   # recent = budget - sink (StreamingLLM)
    beta: float = 20.0     # PyramidKV first : last = 2 beta - 1

    def layer_weights(self, num_layers):
        """Static per-layer weights, or None when budgets follow sparsity."""
        if self.layer_budget == "uniform":
            return [1.0] * num_layers
        if self.layer_budget == "pyramid":
            if num_layers == 1:
                return [1.0]
            last = 1.0 / self.beta
            first = 2.0 - last
            return [first - l * (first - last) / (num_layers - 1) for l in range(num_layers)]
        return None

    def sparsity_in(self, num_layers):
        """The fp32 S_l values that make the budget split follow the static
        weights (None for sparsity-driven budgets)."""
        w = self.layer_weights(num_layers)
        if w is None:
            return None
        top = max(w)
        return [1.0 - x / top for x in w]

    def windows(self, per_layer_budget, recent):
        """(recent, sink) for a round whose per-layer budget is per_layer_budget."""
        if self.window_fills:
            return max(per_layer_budget - self.sink, 0), self.sink
        return recent, self.sink


def get(name, gamma=0.99, sink=0, beta=20.0):
    """The named policy; gamma and sink apply where the policy leaves them free."""
    if name == "lethe":
        return Policy(name, gamma, sink, "sparsity")
    if name == "lethe-shared":
        return Policy(name, gamma, sink, "sparsity", shared=True)
    if name == "h2o":
        return Policy(name, 1.0, 0, "uniform")
    if name == "streaming":
        return Policy(name, 1.0, 4 if sink == 0 else sink, "uniform", window_fills=True)
    if name == "pyramid":
        return Policy(name, gamma, sink, "pyramid", beta=beta)
    raise ValueError("unknown policy %r (one of %s)" % (name, ", ".join(POLICY_NAMES)))


class PruneRound:
    """Device buffers and calls of one prune round of a policy over a cache."""

    def __init__(self, cache, policy):
        import torch
        self.cache, self.policy = cache, policy
        dev = cache.k.device
        Ly, B = cache.L, cache.B
        self.S = torch.empty((B, Ly), dtype=torch.float32, device=dev)
        self.budget = torch.empty((B, Ly), dtype=torch.int32, device=dev)
        self.keep = torch.empty((Ly, cache.rows_per_layer), dtype=torch.uint8, device=dev)
        self.gbud = torch.empty(B, dtype=torch.int64, device=dev)
        self.ws = None  # compaction workspace, allocated by the first eager compaction
        s_in = policy.sparsity_in(Ly)
        self.s_in = None
        if s_in is not None:
            row = torch.tensor(s_in, dtype=torch.float32)
            self.s_in = row[None, :].repeat(B, 1).to(dev)

    def budgets(self, per_layer_budget, recent):
        """Layer sparsity (or the static table) and budgets for a round in
        which sequence b may keep per_layer_budget rows per layer (an int for
        every sequence, one int per sequence, or an int64 device tensor [B]).
        Returns (recent, sink)."""
        import torch
        if isinstance(per_layer_budget, torch.Tensor) and per_layer_budget.is_cuda:
            # Per-sequence budgets already on the device (int64 [B]): no host
            # round trip inside a timed loop.
            if self.policy.window_fills:
                raise ValueError("a window-filling policy needs one host-side budget for every sequence")
            if per_layer_budget.shape != (self.cache.B,):
                raise ValueError("one budget per sequence expected")
            torch.mul(per_layer_budget, self.cache.L, out=self.gbud)
            r, sk = self.policy.windows(0, recent)
            L.layer_sparsity(self.cache, self.gbud, r, sk, self.s_in, self.S, self.budget)
            return r, sk
        if isinstance(per_layer_budget, int):
            per_seq = [per_layer_budget] * self.cache.B
        else:
            per_seq = [int(x) for x in per_layer_budget]
        if len(per_seq) != self.cache.B:
            raise ValueError("one budget per sequence expected")
        if self.policy.window_fills and len(set(per_seq)) > 1:
            raise ValueError("a window-filling policy needs the same budget for every sequence")
        r, sk = self.policy.windows(per_seq[0], recent)
        if len(set(per_seq)) == 1:
            self.gbud.fill_(per_seq[0] * self.cache.L)
        else:
            self.gbud.copy_(torch.tensor([x * self.cache.L for x in per_seq], dtype=torch.int64))
        L.layer_sparsity(self.cache, self.gbud, r, sk, self.s_in, self.S, self.budget)
        return r, sk

    def select(self, recent, sink):
        if self.policy.shared:
            L.rasr_select_shared(self.cache, self.budget, recent, sink, self.keep)
        else:
            L.rasr_select(self.cache, self.budget, recent, sink, self.keep)

    def compact(self):
        if self.ws is None:
            self.ws = self.cache.workspace(L.OP_COMPACT)
        L.kv_compact(self.cache, self.keep, self.ws)

    def plan(self, plan):
        """The compaction as a plan the next decode step of each layer
        carries out (lethe_decode_attn_score_compact)."""
        L.kv_compact_plan(self.cache, self.keep, plan)

    def __call__(self, per_layer_budget, recent):
        r, sk = self.budgets(per_layer_budget, recent)
        self.select(r, sk)
        self.compact()


def per_layer_budget(budget_frac, logical_length):
    """Rows one layer may keep at a round: floor(rho * T) (T the sequence's
    prompt + generated length)."""
    return int(math.floor(budget_frac * logical_length))
