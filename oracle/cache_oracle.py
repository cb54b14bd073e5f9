"""CPU oracle of the mixed-precision expert cache manager (HOBBIT, Section 3.4).

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously correct
reference the library's cache manager is checked against.  Only the test
suite and the CPU-baseline leg of the benchmark may import it; the product
path never calls it.  It shares no code with the library.

What the paper fixes (Section 3.4, "Cache Manager design", Eq. 3)
-----------------------------------------------------------------
* Two caches: one for high-precision expert copies and one for
  low-precision copies, each with its own capacity (counted in experts).
* Records per expert t, kept for the current sequence: R_t, the time
  (token number) of its last use; F_t, how often it was used; H_t, how often
  its high-precision copy was used (not updated by low-precision uses).
  They are updated on every use, hit or miss, and reset when a new
  sequence starts.
* Eq. 3: p_t = w_lru R_t / T + w_lfu F_t / T + w_lhu H_t / T
               + w_fld (1 - ((l_t - l_i + l_n) mod l_n) / l_n),
  with T the current token number, l_i the layer of the expert being
  brought in, l_t the layer of expert t, l_n the number of layers and the
  four weights summing to 1.
* On a miss the expert is brought into the cache of its precision; when
  that cache is full, the resident with the lowest priority relative to
  the incoming expert is evicted.  Experts the predictor marked are masked
  from eviction (Section 3.3).
* Miss penalty (Section 3.4, "Cache replacement policies"): C for a
  high-precision miss, C * B_l / B_h for a low-precision miss (B the bit
  widths).

Readings where the paper is silent (also listed in the design notes)
-------------------------------------------------------------------
* An expert is the pair (layer, expert index); a use names the copy used
  (high or low) and is a hit when that copy is resident in its cache.
* Tokens are numbered 1, 2, ... from the start of the sequence; before
  the first token (T = 0) the three record terms are taken as 0.
* Ties in priority evict the resident with the smallest key
  layer * n_experts + expert.
* If every resident of the full cache is masked, the lowest-priority masked
  resident is evicted (the use is never refused).
* The incoming expert is always inserted (the paper replaces the
  lowest-priority resident with it).
* Eq. 3's terms are evaluated in double precision in the order written.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass
class CacheConfig:
    n_layers: int
    n_experts: int
    hi_capacity: int
    lo_capacity: int
    w_lru: float
    w_lfu: float
    w_lhu: float
    w_fld: float
    bits_hi: int = 16
    bits_lo: int = 4
    miss_cost: float = 1.0   # C: cost of loading one high-precision expert


@dataclass
class CacheOracle:
    cfg: CacheConfig
    T: int = 0
    R: dict = field(default_factory=dict)
    F: dict = field(default_factory=dict)
    H: dict = field(default_factory=dict)
    resident: tuple = field(default_factory=lambda: (set(), set()))  # (high, low)
    masked: set = field(default_factory=set)
    penalty: float = 0.0
    hi_misses: int = 0
    lo_misses: int = 0
    hits: int = 0

    # ---- sequence and token boundaries ------------------------------------
    def begin_sequence(self):
        """A new sequence: the LRU, LFU and LHU records restart (Section 3.4);
        the cache contents stay."""
        self.T = 0
        self.R.clear()
        self.F.clear()
        self.H.clear()

    def begin_token(self):
        self.T += 1

    # ---- Eq. 3 --------------------------------------------------------------
    def priority(self, t, layer_i: int) -> float:
        c = self.cfg
        l_t = t[0]
        if self.T > 0:
            p_lru = self.R.get(t, 0) / self.T
            p_lfu = self.F.get(t, 0) / self.T
            p_lhu = self.H.get(t, 0) / self.T
        else:
            p_lru = p_lfu = p_lhu = 0.0
        p_fld = 1.0 - ((l_t - layer_i + c.n_layers) % c.n_layers) / c.n_layers
        return c.w_lru * p_lru + c.w_lfu * p_lfu + c.w_lhu * p_lhu + c.w_fld * p_fld

    def victim(self, cache: set, layer_i: int):
        """Lowest-priority resident (unmasked ones first), ties to the smaller
        key layer * n_experts + expert."""
        E = self.cfg.n_experts
        pool = [t for t in cache if t not in self.masked] or list(cache)
        return min(pool, key=lambda t: (self.priority(t, layer_i), t[0] * E + t[1]))

    # ---- one use of an expert ----------------------------------------------
    def access(self, layer: int, expert: int, high: bool):
        """Use of expert (layer, expert) through its high (True) or low copy.
        Returns (hit, evicted) with evicted = (layer, expert) or None."""
        c = self.cfg
        t = (layer, expert)
        # the records are updated on every use (the LHU record only for
        # high-precision uses)
        self.R[t] = self.T
        self.F[t] = self.F.get(t, 0) + 1
        if high:
            self.H[t] = self.H.get(t, 0) + 1
        cache = self.resident[0] if high else self.resident[1]
        cap = c.hi_capacity if high else c.lo_capacity
        if t in cache:
            self.hits += 1
            return True, None
        if high:
            self.hi_misses += 1
            self.penalty += c.miss_cost
        else:
            self.lo_misses += 1
            self.penalty += c.miss_cost * c.bits_lo / c.bits_hi
        evicted = None
        if cap <= 0:
            return False, None
        if len(cache) >= cap:
            evicted = self.victim(cache, layer)
            cache.remove(evicted)
        cache.add(t)
        return False, evicted

    def set_mask(self, layer: int, expert: int, on: bool):
        if on:
            self.masked.add((layer, expert))
        else:
            self.masked.discard((layer, expert))

    def clear_masks(self):
        self.masked.clear()

    def contains(self, layer: int, expert: int, high: bool) -> bool:
        return (layer, expert) in (self.resident[0] if high else self.resident[1])


def replay(cfg: CacheConfig, trace, sequence_starts=()):
    """Replay a trace of (token, layer, expert, high) uses through a fresh
    oracle; the token number advances whenever it changes, a new sequence
    starts at every index in sequence_starts.  Returns the oracle and the
    per-use (hit, evicted) list."""
    o = CacheOracle(cfg)
    starts = set(sequence_starts)
    out = []
    last_tok = None
    for i, (tok, layer, expert, high) in enumerate(trace):
        if i in starts:
            o.begin_sequence()
            last_tok = None
        if tok != last_tok:
            o.begin_token()
            last_tok = tok
        out.append(o.access(layer, expert, bool(high)))
    return o, out
