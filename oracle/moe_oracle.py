"""CPU oracle of the mixed-precision MoE layer (HOBBIT, arXiv 2411.01433).

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously correct
reference that the HIP library is checked against.  Only the test suite,
the smoke check and the CPU-baseline leg of the benchmark may import it;
the product path never calls it.  It shares no code with the HIP side.

Everything is computed in float64 from the fp16 inputs (which upcast
exactly).  Each function cites the passage of the paper it follows.

What the paper fixes and what is a reading
------------------------------------------
* Eq. 1 (Section 2.1): y = sum_i G(x)_{e_i} E_{e_i}(x) over the K selected
  experts; G is a linear layer followed by top-k.
* Section 3.2: the selected gate values are normalised; they are ranked in
  descending order, Eq. 2 gives the unimportance score s, threshold T1
  splits high from low precision, T2 marks experts to skip, and the first
  (largest-gate) expert is always high precision.
* Readings where the paper is silent (also listed in the design notes):
  - normalisation = softmax over the K selected logits;
  - expert FFN = SwiGLU without bias, W2 (silu(W1 x) * (W3 x));
  - low-precision copy = symmetric signed integer, group of 32 consecutive
    weights along the input dimension, one fp16 scale per group (the int8
    high-precision copy of an int8 model, Section 4.1, is the same
    quantiser at b = 8),
    s = fp16_rne(max|w| / qmax), q = clamp(rne(w / s), -2^(b-1), qmax),
    qmax = 2^(b-1) - 1; stored offset-binary u = q + 2^(b-1), packed
    little-endian within each byte;
  - exact ties: lower expert index (top-k) / lower slot (ranking) first;
  - a skipped expert contributes zero and the rest are not renormalised;
  - stacks: pre-norm residual h <- h + MoE(fp16(rmsnorm(h))), no gain,
    eps = 1e-5.

Parity pinning: every function here is pinned by the CPU tests against
brute force, closed forms, library routines or hand-worked examples.
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass

import numpy as np

# precision classes of one (token, slot) assignment
PREC_HIGH = 0   # high-precision copy (fp16; int8 for the int8-model tags)
PREC_LOW = 1    # low-precision copy (int4 or int2, from the expert's tag)
PREC_SKIP = 2   # expert bypassed (second threshold T2)

# per-expert tags: state of the expert in the (simulated) expert cache
TAG_FP16 = 0       # resident at full precision: always high
TAG_INT4 = 1       # resident as int4 copy: always low (4 bit)
TAG_INT2 = 2       # resident as int2 copy: always low (2 bit)
TAG_MISS_INT4 = 3  # cache miss, low copy is int4: Eq. 2 rule decides
TAG_MISS_INT2 = 4  # cache miss, low copy is int2: Eq. 2 rule decides
# int8 model (Section 4.1: int2 copies replace int8 experts): the high copy
# is the expert's int8 quantisation
TAG_INT8 = 5            # resident as int8 copy: always high (8 bit)
TAG_MISS_INT8_INT2 = 6  # cache miss, int8 high / int2 low: Eq. 2 rule decides

GROUP = 32
RMS_EPS = 1e-5


def low_bits_of_tag(tag: int) -> int:
    """Bit width of the low-precision copy an expert tag refers to (Section 4.1
    Configurations: int4 replaces fp16, int2 replaces int8)."""
    return {TAG_FP16: 0, TAG_INT4: 4, TAG_INT2: 2,
            TAG_MISS_INT4: 4, TAG_MISS_INT2: 2,
            TAG_INT8: 0, TAG_MISS_INT8_INT2: 2}[int(tag)]


def high_bits_of_tag(tag: int) -> int:
    """Bit width of the high-precision copy: 16 (fp16 model) or 8 (int8
    model, Section 4.1)."""
    return 8 if int(tag) in (TAG_INT8, TAG_MISS_INT8_INT2) else 16


# --------------------------------------------------------------------------
# Gating: Eq. 1 and Section 2.1 ("a linear layer followed by a Top-k").
# --------------------------------------------------------------------------
def router_logits(x16: np.ndarray, wg16: np.ndarray) -> np.ndarray:
    """l[t, e] = sum_d x[t, d] * Wg[e, d]  (gating linear layer, Eq. 1)."""
    x = np.asarray(x16, dtype=np.float64)
    wg = np.asarray(wg16, dtype=np.float64)
    return x @ wg.T


def topk(logits_row: np.ndarray, k: int) -> np.ndarray:
    """Indices of the K largest logits, largest first; exact ties go to the
    lower expert index (Section 2.1 top-k)."""
    order = sorted(range(len(logits_row)), key=lambda e: (-logits_row[e], e))
    return np.array(order[:k], dtype=np.int64)


def gate_weights(selected_logits: np.ndarray) -> np.ndarray:
    """Normalised gate values of the selected experts (Section 3.2: values are
    normalised): softmax over the K selected logits."""
    z = np.asarray(selected_logits, dtype=np.float64)
    ez = np.exp(z - z.max())
    return ez / ez.sum()


# --------------------------------------------------------------------------
# Token-level precision decision: Section 3.2, Eq. 2.
# --------------------------------------------------------------------------
def importance_rank(w: np.ndarray) -> np.ndarray:
    """Slots ordered by descending gate weight (ties: lower slot first)."""
    return np.array(sorted(range(len(w)), key=lambda j: (-w[j], j)),
                    dtype=np.int64)


def unimportance_scores(w: np.ndarray) -> np.ndarray:
    """Eq. 2: after ranking the K experts by descending gate value, the score
    of the expert at rank i is the sum of the gate values ranked above it,
    and 0 for rank 0.  Returned per slot (not per rank)."""
    order = importance_rank(w)
    s = np.zeros(len(w), dtype=np.float64)
    running = 0.0
    for i, slot in enumerate(order):
        s[slot] = 0.0 if i == 0 else running
        running += float(w[slot])
    return s


def precision_from_score(score: float, rank: int, t1: float, t2: float) -> int:
    """Section 3.2 thresholds: s <= T1 -> high; T1 < s <= T2 -> low;
    s > T2 -> skip; the rank-0 expert is always high."""
    if rank == 0 or score <= t1:
        return PREC_HIGH
    if score <= t2:
        return PREC_LOW
    return PREC_SKIP


def token_precisions(w: np.ndarray, sel: np.ndarray, tags: np.ndarray,
                     t1: float, t2: float) -> np.ndarray:
    """Precision class of every slot of one token.  Experts whose tag says
    they are resident (hit) run at the precision they are held in; for a
    cache-miss tag the Eq. 2 rule decides (Section 3.2, Fig. 6 flow)."""
    s = unimportance_scores(w)
    order = importance_rank(w)
    rank_of = np.empty(len(w), dtype=np.int64)
    rank_of[order] = np.arange(len(w))
    out = np.empty(len(w), dtype=np.int64)
    for j, e in enumerate(sel):
        tag = int(tags[e])
        if tag in (TAG_FP16, TAG_INT8):
            out[j] = PREC_HIGH
        elif tag in (TAG_INT4, TAG_INT2):
            out[j] = PREC_LOW
        else:
            out[j] = precision_from_score(s[j], int(rank_of[j]), t1, t2)
    return out


# --------------------------------------------------------------------------
# Low-precision copies: group-wise symmetric quantisation (Section 2.2 and
# Section 4.1 Configurations; format is a reading, see module docstring).
# --------------------------------------------------------------------------
def _round_half_even(v: np.ndarray) -> np.ndarray:
    return np.round(v)  # numpy rounds half to even


def quantize(w16: np.ndarray, bits: int, group: int = GROUP):
    """Quantise a matrix [rows, cols] group-wise along columns.  The weights
    are fp16 in use; any float input is taken at its exact value.

    Returns (q, scales): q int64 [rows, cols] in [-2^(b-1), 2^(b-1)-1],
    scales fp16 [rows, cols/group].
    """
    w = np.asarray(w16).astype(np.float64)
    rows, cols = w.shape
    assert cols % group == 0
    qmax = 2 ** (bits - 1) - 1
    qmin = -(2 ** (bits - 1))
    g = w.reshape(rows, cols // group, group)
    m = np.abs(g).max(axis=2)                       # absmax per group
    s16 = (m / qmax).astype(np.float16)             # one RNE rounding to fp16
    s = s16.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(s[..., None] > 0, g / s[..., None], 0.0)
    q = np.clip(_round_half_even(r), qmin, qmax).astype(np.int64)
    return q.reshape(rows, cols), s16


def dequantize(q: np.ndarray, s16: np.ndarray, group: int = GROUP) -> np.ndarray:
    """w_hat = q * s per group, in float64 (exact)."""
    rows, cols = q.shape
    s = np.asarray(s16, dtype=np.float16).astype(np.float64)
    return (q.reshape(rows, cols // group, group).astype(np.float64)
            * s[..., None]).reshape(rows, cols)


def pack_codes(q: np.ndarray, bits: int) -> np.ndarray:
    """Offset-binary codes u = q + 2^(b-1), packed little-endian: element j of
    a row sits at bit b * (j mod (8/b)) of byte floor(j * b / 8)."""
    rows, cols = q.shape
    per = 8 // bits
    u = (q + 2 ** (bits - 1)).astype(np.uint8)
    u = u.reshape(rows, cols // per, per)
    out = np.zeros((rows, cols // per), dtype=np.uint8)
    for j in range(per):
        out |= (u[:, :, j] << (bits * j)).astype(np.uint8)
    return out


def unpack_codes(packed: np.ndarray, bits: int) -> np.ndarray:
    """Inverse of pack_codes: packed u8 [rows, cols*b/8] -> q int64."""
    rows, nb = packed.shape
    per = 8 // bits
    mask = (1 << bits) - 1
    u = np.empty((rows, nb, per), dtype=np.int64)
    for j in range(per):
        u[:, :, j] = (packed.astype(np.int64) >> (bits * j)) & mask
    return u.reshape(rows, nb * per) - 2 ** (bits - 1)


@dataclass
class LowCopy:
    """One matrix's low-precision copy: packed codes and fp16 group scales."""
    bits: int
    codes: np.ndarray   # uint8 [rows, cols*bits/8]
    scales: np.ndarray  # float16 [rows, cols/32]

    def dense(self) -> np.ndarray:
        return dequantize(unpack_codes(self.codes, self.bits), self.scales)


def make_low_copy(w16: np.ndarray, bits: int) -> LowCopy:
    q, s = quantize(w16, bits)
    return LowCopy(bits, pack_codes(q, bits), s)


# --------------------------------------------------------------------------
# Expert FFN (Section 2.1: FFN experts; SwiGLU reading) and Eq. 1 combine.
# --------------------------------------------------------------------------
def silu(a: np.ndarray) -> np.ndarray:
    return a / (1.0 + np.exp(-a))


def swiglu_hidden(x: np.ndarray, w1: np.ndarray, w3: np.ndarray) -> np.ndarray:
    """h = silu(W1 x) * (W3 x); x [n, d], W1/W3 [f, d] -> h [n, f] (float64)."""
    a = x @ w1.T
    b = x @ w3.T
    return silu(a) * b


def swiglu_expert(x: np.ndarray, w1: np.ndarray, w3: np.ndarray,
                  w2: np.ndarray) -> np.ndarray:
    """E(x) = W2 (silu(W1 x) * (W3 x)); W2 [d, f] -> [n, d] (float64)."""
    return swiglu_hidden(x, w1, w3) @ w2.T


@dataclass
class Expert:
    """fp16 weights of one expert plus the low-precision copy it may use."""
    w1: np.ndarray  # fp16 [f, d]
    w3: np.ndarray  # fp16 [f, d]
    w2: np.ndarray  # fp16 [d, f]
    tag: int = TAG_FP16

    def weights(self, prec: int):
        """float64 weights at the requested precision class (memoised)."""
        memo = self.__dict__.setdefault("_memo", {})
        if prec not in memo:
            if prec == PREC_HIGH and high_bits_of_tag(self.tag) == 8:
                memo[prec] = tuple(make_low_copy(w, 8).dense()
                                   for w in (self.w1, self.w3, self.w2))
            elif prec == PREC_HIGH:
                memo[prec] = (self.w1.astype(np.float64), self.w3.astype(np.float64),
                              self.w2.astype(np.float64))
            else:
                bits = low_bits_of_tag(self.tag)
                assert bits in (2, 4), "low precision requested for an fp16-only expert"
                memo[prec] = tuple(make_low_copy(w, bits).dense()
                                   for w in (self.w1, self.w3, self.w2))
        return memo[prec]


@dataclass
class Routing:
    idx: np.ndarray     # int64 [T, K], slot 0 = largest logit
    w: np.ndarray       # float64 [T, K]
    prec: np.ndarray    # int64 [T, K] PREC_*
    logits: np.ndarray  # float64 [T, E]


def route(x16: np.ndarray, wg16: np.ndarray, tags, k: int,
          t1: float, t2: float, forced_idx: np.ndarray | None = None) -> Routing:
    """Gating + top-k + normalisation + Eq. 2 decision for every token.
    ``forced_idx`` replaces the top-k choice for tokens flagged as near-ties
    by the comparison (the selected set then comes from the implementation
    under test)."""
    l = router_logits(x16, wg16)
    T = l.shape[0]
    idx = np.zeros((T, k), dtype=np.int64)
    w = np.zeros((T, k), dtype=np.float64)
    prec = np.zeros((T, k), dtype=np.int64)
    tags = np.asarray(tags)
    for t in range(T):
        sel = topk(l[t], k) if forced_idx is None else np.asarray(forced_idx[t])
        idx[t] = sel
        w[t] = gate_weights(l[t, sel])
        prec[t] = token_precisions(w[t], sel, tags, t1, t2)
    return Routing(idx, w, prec, l)


def layer_output(x16: np.ndarray, experts, r: Routing) -> np.ndarray:
    """Eq. 1 for given routing decisions: y[t] = sum_k w[t,k] * E_{idx[t,k]}(x[t])
    with each expert at the precision class r.prec chose; a skipped term is
    zero.  ``experts[e]`` yields an Expert (it may be built on demand)."""
    x = np.asarray(x16, dtype=np.float64)
    T, d = x.shape
    y = np.zeros((T, d), dtype=np.float64)
    cache = {}
    for t in range(T):
        for j in range(r.idx.shape[1]):
            p = int(r.prec[t, j])
            if p == PREC_SKIP:
                continue
            e = int(r.idx[t, j])
            if (e, p) not in cache:
                cache[(e, p)] = experts[e].weights(p)
            w1, w3, w2 = cache[(e, p)]
            y[t] += r.w[t, j] * swiglu_expert(x[t:t + 1], w1, w3, w2)[0]
    return y


def layer_forward(x16: np.ndarray, wg16: np.ndarray, experts, k: int,
                  t1: float, t2: float, forced_idx=None):
    """Eq. 1 with the Section 3.2 decisions: route, then layer_output.
    Returns (y, routing) with y float64 [T, d]."""
    tags = [e.tag for e in experts]
    r = route(x16, wg16, tags, k, t1, t2, forced_idx)
    return layer_output(x16, experts, r), r


# --------------------------------------------------------------------------
# Stack glue (reading: Mixtral-style pre-norm residual between MoE layers).
# --------------------------------------------------------------------------
def rmsnorm(h: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    h = np.asarray(h, dtype=np.float64)
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)


def residual_step(h: np.ndarray, y: np.ndarray, eps: float = RMS_EPS):
    """h' = h + y; x' = fp16(rmsnorm(h')).  Returns (h', x' fp16)."""
    h2 = np.asarray(h, dtype=np.float64) + np.asarray(y, dtype=np.float64)
    return h2, rmsnorm(h2, eps).astype(np.float16)


# --------------------------------------------------------------------------
# Adaptive Expert Predictor: the Stacking Computer (Section 3.3, "Expert
# predictor design", Fig. 7).
# --------------------------------------------------------------------------
@dataclass
class Prediction:
    idx: np.ndarray      # [T, p, K] predicted experts of layers l+1 .. l+p
    w: np.ndarray        # [T, p, K] their normalised gate values
    logits: np.ndarray   # [T, p, E]
    first_miss: int      # first j in 1..p with a predicted expert not cached; 0 if none
    preload: int         # bitmask of the predicted experts of layer first_miss not cached


def predict_next_layers(x16: np.ndarray, wg16_next, cached, k: int,
                        forced_idx: np.ndarray | None = None) -> Prediction:
    """Predicted experts of the next p layers from the current layer's gating
    input (Section 3.3): gating inputs of consecutive layers are similar, so
    the gate of layer l+j applied to layer l's input predicts layer l+j's
    choice; each prediction uses that layer's own top-k and normalisation.
    Walking j = 1, 2, ..., p, prediction continues while every predicted
    expert of layer l+j is in the expert cache and stops at the first layer
    with a missing one, whose missing experts are the ones to preload.
    ``cached[j-1]`` is the bitmask of layer l+j's cached experts.  The
    Stacking Computer evaluates the p gates as one stacked product; here
    they are p independent routers.  ``forced_idx`` [T, p, K] replaces the
    top-k choice where the comparison flagged a near-tie."""
    x = np.asarray(x16)
    p = len(wg16_next)
    T = x.shape[0]
    E = np.asarray(wg16_next[0]).shape[0]
    idx = np.zeros((T, p, k), dtype=np.int64)
    w = np.zeros((T, p, k), dtype=np.float64)
    logits = np.zeros((T, p, E), dtype=np.float64)
    for j in range(p):
        l = router_logits(x, wg16_next[j])
        logits[:, j] = l
        for t in range(T):
            sel = topk(l[t], k) if forced_idx is None else np.asarray(forced_idx[t, j])
            idx[t, j] = sel
            w[t, j] = gate_weights(l[t, sel])
    first, pre = 0, 0
    for j in range(p):
        need = 0
        for e in idx[:, j].ravel():
            need |= 1 << int(e)
        miss = need & ~int(cached[j])
        if miss:
            first, pre = j + 1, miss
            break
    return Prediction(idx, w, logits, first, pre)


# --------------------------------------------------------------------------
# Brute-force variants (pure Python loops) used to pin the above.
# --------------------------------------------------------------------------
def brute_router_logits(x16, wg16):
    x = np.asarray(x16, dtype=np.float64)
    wg = np.asarray(wg16, dtype=np.float64)
    T, d = x.shape
    E = wg.shape[0]
    out = np.zeros((T, E))
    for t in range(T):
        for e in range(E):
            acc = 0.0
            for i in range(d):
                acc += float(x[t, i]) * float(wg[e, i])
            out[t, e] = acc
    return out


def brute_topk_set(logits_row, k):
    """The K-subset every member of which is >= every non-member (exhaustive
    search over all C(E, K) subsets; the lowest-index subset among ties)."""
    E = len(logits_row)
    for sub in itertools.combinations(range(E), k):
        rest = [e for e in range(E) if e not in sub]
        if all(logits_row[a] > logits_row[b] or
               (logits_row[a] == logits_row[b] and a < b)
               for a in sub for b in rest):
            return set(sub)
    raise AssertionError("no top-k subset found")


def brute_nearest_code(w: float, s: float, bits: int) -> int:
    """Nearest representable level q*s over all 2^b codes (ties to even q)."""
    if s == 0.0:
        return 0
    best = None
    for q in range(-(2 ** (bits - 1)), 2 ** (bits - 1)):
        err = abs(w - q * s)
        key = (err, q % 2, q)
        if best is None or key < best[0]:
            best = (key, q)
    return best[1]


def brute_expert(x_row, w1, w3, w2):
    """E(x) for one token by explicit loops (float64)."""
    w1 = np.asarray(w1, dtype=np.float64)
    w3 = np.asarray(w3, dtype=np.float64)
    w2 = np.asarray(w2, dtype=np.float64)
    f, d = w1.shape
    h = [0.0] * f
    for r in range(f):
        a = sum(float(w1[r, i]) * float(x_row[i]) for i in range(d))
        b = sum(float(w3[r, i]) * float(x_row[i]) for i in range(d))
        h[r] = a / (1.0 + np.exp(-a)) * b
    out = np.zeros(w2.shape[0])
    for o in range(w2.shape[0]):
        out[o] = sum(float(w2[o, r]) * h[r] for r in range(f))
    return out
