"""Seeded synthetic expert-use traces for the cache manager.

Stand-in for the routing traces of real prompts (the paper's Fig. 10
statistics come from Mixtral / Phi-MoE on real data, not available here).
The generator only draws expert ids; it computes nothing of the method:
* per sequence and layer, a preference order of the experts drawn by a
  seeded permutation, with Zipf-like weights (sequence-level preferences,
  Fig. 10b);
* with probability p_repeat a token's first expert at a layer repeats the
  previous token's first expert there (temporal reuse, Fig. 10a);
* slot 0 is used through its high-precision copy, slot k > 0 through its
  high copy with a per-sequence propensity of that (layer, expert) drawn
  uniformly from [0, 2 p_high] (experts differ in how often their high copy
  is used, Fig. 11a), else its low copy (a stand-in for the token-level
  rule of Eq. 2, which needs real gate values).
A use is (token, layer, expert, high); uses of a token are listed layer by
layer, slot by slot.
"""
from __future__ import annotations

import numpy as np


def expert_trace(seed: int, n_seqs: int, seq_len: int, n_layers: int, n_experts: int,
                 top_k: int = 2, p_repeat: float = 0.4, zipf: float = 1.0,
                 p_high: float = 0.5):
    """Returns (tokens, layers, experts, highs, new_sequence) int32 / uint8 arrays."""
    rng = np.random.default_rng(seed)
    toks, lays, exps, highs, news = [], [], [], [], []
    w = 1.0 / np.arange(1, n_experts + 1) ** zipf
    w /= w.sum()
    tok = 0
    for s in range(n_seqs):
        order = np.stack([rng.permutation(n_experts) for _ in range(n_layers)])
        ph = rng.uniform(0.0, min(1.0, 2.0 * p_high), size=(n_layers, n_experts))
        prev = np.full(n_layers, -1)
        first = True
        for t in range(seq_len):
            tok += 1
            for layer in range(n_layers):
                chosen = []
                if prev[layer] >= 0 and rng.random() < p_repeat:
                    chosen.append(int(prev[layer]))
                while len(chosen) < top_k:
                    e = int(order[layer][rng.choice(n_experts, p=w)])
                    if e not in chosen:
                        chosen.append(e)
                prev[layer] = chosen[0]
                for k, e in enumerate(chosen):
                    toks.append(tok)
                    lays.append(layer)
                    exps.append(e)
                    highs.append(1 if k == 0 or rng.random() < ph[layer][e] else 0)
                    news.append(1 if first else 0)
                    first = False
    return (np.array(toks, np.int32), np.array(lays, np.int32), np.array(exps, np.int32),
            np.array(highs, np.int32), np.array(news, np.uint8))
