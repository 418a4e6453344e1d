"""Low-overhead compensation (oracle, fp64) -- Sec. IV-C.

Test infrastructure only; see the package docstring.

Step 1 masks every expert outside A_trans; step 2 takes a top-k of what is
left, so the weight of pruned experts moves onto experts that are executed
anyway.  Reading taken: a token keeps every expert of its own K_t that
survived pruning, and only the freed slots are refilled, from A_trans minus
K_t, best router key first (ties to the lower index), with no group limit.
This keeps a layer without pruning identical to the plain layer, and never
drops a token's expert whose gate weight reached the threshold.  When
A_trans has fewer than k experts the token gets fewer than k (padded with
id -1, weight 0).  Final weights are the router scores renormalised over
K_final and multiplied by the routed scaling factor, so the gate mass is
conserved.
"""
from __future__ import annotations

import numpy as np

# Ablation variants of the refill (the paper contrasts its score-based
# compensation with a random selection among the cheap experts):
#   "score"  - the paper's mechanism, as described above;
#   "none"   - no refill: K_final = K_t within A_trans, weights renormalised;
#   "random" - the freed slots take the experts of A_trans minus K_t with the
#              largest counter-based random keys (below), lower index on ties;
#   "literal" - Sec. IV-C's second step read literally: K_final is the top-k
#              of the masked router keys, i.e. the k best keys of A_trans
#              (ties to the lower index), whether or not they were in K_t and
#              with no group limit.  It can drop a token's own surviving
#              expert for a better-keyed one from a group the token did not
#              select, so unlike "score" it does not reduce to the plain layer
#              when nothing is pruned (unless A_trans lies within the token's
#              groups, as at T = 1).
_M64 = (1 << 64) - 1
_GOLDEN_GAMMA = 0x9E3779B97F4A7C15


def splitmix64(state: int) -> int:
    """The output SplitMix64 (Steele, Lea and Flood, OOPSLA 2014, in the
    64-bit form Vigna publishes) produces from `state`: add the golden
    gamma, then two xor-shift-multiply rounds and a final xor-shift."""
    z = (state + _GOLDEN_GAMMA) & _M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


def refill_key(seed: int, t: int, e: int, E: int) -> int:
    """53-bit random key of (token t, expert e) for the random refill: the
    SplitMix64 output of counter (seed << 32) | (t * E + e), top 53 bits."""
    return splitmix64(((int(seed) & 0xFFFFFFFF) << 32) | (int(t) * int(E) + int(e))) >> 11


def compensate_token(key: np.ndarray, s: np.ndarray, orig_ids, trans: np.ndarray,
                     k: int, routed_scaling: float, refill: str = "score", seed: int = 0, t: int = 0):
    """Return (ids, w) for one token: K_final in rank order (key desc, index
    asc) and w_e = routed_scaling * s_e / sum_{K_final} s (float64).
    `refill`, `seed` and the token index `t` select the ablation variant."""
    orig = list(orig_ids)
    if refill == "literal":
        final = sorted(np.flatnonzero(trans).tolist(), key=lambda e: (-float(key[e]), e))[:k]
        total = 0.0
        for e in final:
            total += float(s[e])
        w = [float(routed_scaling) * (float(s[e]) / total) for e in final]
        return final, w, sum(1 for e in final if e not in orig)
    keep = [e for e in orig if trans[e]]
    pool = [e for e in np.flatnonzero(trans).tolist() if e not in orig]
    if refill == "score":
        pool.sort(key=lambda e: (-float(key[e]), e))
    elif refill == "random":
        E = len(trans)
        pool.sort(key=lambda e: (-refill_key(seed, t, e, E), e))
    elif refill == "none":
        pool = []
    else:
        raise ValueError(refill)
    refill = pool[:max(0, k - len(keep))]
    final = sorted(keep + refill, key=lambda e: (-float(key[e]), e))
    total = 0.0
    for e in final:
        total += float(s[e])
    w = [float(routed_scaling) * (float(s[e]) / total) for e in final]
    return final, w, len(refill)


def compensate_batch(keys: np.ndarray, s: np.ndarray, orig_ids: np.ndarray,
                     trans: np.ndarray, k: int, routed_scaling: float, refill: str = "score", seed: int = 0):
    """Compensation for every token.  Returns (ids [T][k] int, -1 padded;
    w [T][k] float64, 0 padded; total refilled slots)."""
    T = orig_ids.shape[0]
    ids = -np.ones((T, k), dtype=np.int64)
    w = np.zeros((T, k), dtype=np.float64)
    n_refill = 0
    for t in range(T):
        fid, fw, nr = compensate_token(keys[t], s[t], orig_ids[t], trans, k, routed_scaling, refill, seed, t)
        ids[t, :len(fid)] = fid
        w[t, :len(fw)] = fw
        n_refill += nr
    return ids, w, n_refill
