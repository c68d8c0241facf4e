"""ORACLE — test infrastructure, not part of the product.

The co-activation predictor of WiSP (arXiv 2606.21868, App. E), written from its definition in
exact rational arithmetic (``fractions.Fraction``), so that equal scores are equal and every order
is exact:

- A[(l, l')][(e, e')] counts the forward passes in which expert e fired at layer l and expert e'
  at the later layer l' (App. E, "Construction");
- P_{l,l'}(e' | e) = A(e, e') / sum_j A(e, j), the count normalised by the source marginal;
- s_{l'}(e') = sum over earlier layers l routed in the current pass of gamma^(l' - l) times
  sum over e in R_l of P_{l,l'}(e' | e);
- the prediction is the highest-scoring experts, ordered (score desc, id asc), positive scores only.

``horizon`` keeps the source layers with l' - l <= horizon (None keeps every earlier layer, as the
paper's sum does).  The tables start empty and learn online: a pass's routed sets are counted when
the pass ends.  Only ``tests/`` may import this module.
"""
from __future__ import annotations

from collections import defaultdict
from fractions import Fraction


class CoActivation:
    def __init__(self, n_layers, n_experts, horizon=None, gamma=Fraction(1)):
        self.L = n_layers
        self.N = n_experts
        self.horizon = horizon
        self.gamma = Fraction(gamma)
        self.A = defaultdict(lambda: defaultdict(int))   # (l, l') -> {(e, e'): count}
        self.R = {}                                      # layer -> set of experts, current pass

    def _in_horizon(self, l, lt):
        return l < lt and (self.horizon is None or lt - l <= self.horizon)

    def observe(self, layer, ids):
        self.R[layer] = set(int(e) for e in ids)

    def end_pass(self):
        for l, src in self.R.items():
            for lt, tgt in self.R.items():
                if not self._in_horizon(l, lt):
                    continue
                tab = self.A[(l, lt)]
                for e in src:
                    for et in tgt:
                        tab[(e, et)] += 1
        self.R = {}

    def marginal(self, l, lt, e):
        """sum_j A_{l,l'}(e, j): how often e at l co-fired with anything at l'."""
        return sum(c for (a, _), c in self.A[(l, lt)].items() if a == e)

    def conditional(self, l, lt, e, et):
        """P_{l,l'}(e' | e), or None if e never fired at l in a counted pass."""
        m = self.marginal(l, lt, e)
        if m == 0:
            return None
        return Fraction(self.A[(l, lt)].get((e, et), 0), m)

    def scores(self, layer):
        """s_layer(e') for every candidate e' (exact)."""
        s = [Fraction(0)] * self.N
        for l, src in self.R.items():
            if not self._in_horizon(l, layer):
                continue
            w = self.gamma ** (layer - l)
            tab = self.A[(l, layer)]
            for e in src:
                m = self.marginal(l, layer, e)
                if m == 0:
                    continue
                for et in range(self.N):
                    c = tab.get((e, et), 0)
                    if c:
                        s[et] += w * Fraction(c, m)
        return s

    def predict(self, layer, depth):
        s = self.scores(layer)
        cand = [e for e in range(self.N) if s[e] > 0]
        cand.sort(key=lambda e: (-s[e], e))
        return cand[:depth], [s[e] for e in cand[:depth]]
