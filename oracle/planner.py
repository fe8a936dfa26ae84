"""Independent CPU CQS planner (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

What it follows
---------------
* Section 3: a sequence is split into c = l(l-1)+1 chunks; subsequence i is
  the concatenation of chunks (i + o) mod c for o in the interest set I.
* App. C (Table "interest_set"): I is a perfect (c, l, 1) cyclic difference
  set; its paired set is (0, 1, c+1-a_{l-1}, ..., c+1-a_2).
* Section 3.3: subsequence i keeps the diagonal chunk pair (i, i) and masks
  the other diagonal pairs it holds; depth itr gives c**itr subsequences, each
  re-partitioned and inheriting the masks of the levels above.
* Alg. 3 (BuildSubseq): per quorum tuple (q_1..q_itr) in lexicographic order,
  re-chunk the current token list at every level, keep the chunks
  {(q_t + o) mod c}, and record, for every chunk other than the owner q_t, the
  group of local tokens that came from it.  Two local tokens are masked from
  each other iff some recorded group holds both.
* App. A.2: each token carries group bits; local pair (q, k) is kept iff
  bits[q] & bits[k] == 0.  Per 64-token block the OR and AND of the bits are
  stored; a 128x128 tile is clear if OR(rows) & OR(cols) == 0, fully masked if
  AND(rows) & AND(cols) != 0, and mixed otherwise.

Readings where the paper is silent or inconsistent
--------------------------------------------------
1. BalancedChunkLayout(L, c): the first (L mod c) chunks hold floor(L/c)+1
   tokens, the rest floor(L/c) (the numpy.array_split rule).
2. Chunks inside a task are gathered in ascending chunk order, so local token
   order equals global order (App. A.3); Alg. 3 says "ordered by I".  Both
   give the same kept pair set; ascending lets plain causal masking compose.
3. Group bit numbering: at level t (1-based) the chunk (q_t + I[j]) mod c,
   j = 1..l-1, gets bit (t-1)*(l-1) + (j-1).  Alg. 3's Unique only merges
   groups with identical token sets, which cannot change the mask.
4. Causal attention keeps a pair iff the key's global index <= the query's.
5. Section 3.3 allows a different valid interest set at each depth.  With
   level t using (c_t, I_t), the quorum tuple ranges over c_1 x ... x c_itr
   (lexicographic), level t re-chunks into c_t chunks, and its non-owner
   chunks take bits s_t + (j-1), where s_t is the sum of (l_u - 1) over the
   levels u above t (reading 3 is the case of equal levels).
"""
import itertools

import numpy as np

# Table "interest_set" (App. C): examples for several l.  c = l(l-1)+1.
PAPER_INTEREST_SETS = {
    7: (0, 1, 3),
    13: (0, 1, 3, 9),
    21: (0, 1, 4, 14, 16),
    31: (0, 1, 3, 8, 12, 18),
    57: (0, 1, 3, 13, 32, 36, 43, 52),
    73: (0, 1, 3, 7, 15, 31, 36, 54, 63),
    91: (0, 1, 3, 9, 27, 49, 56, 61, 77, 81),
    133: (0, 1, 3, 12, 20, 34, 38, 81, 88, 94, 104, 109),
}


def is_perfect_difference_set(I, c):
    """True iff every nonzero residue mod c occurs exactly once among the
    differences x - y (x != y) of I (App. C, lambda = 1)."""
    counts = np.zeros(c, dtype=np.int64)
    for x in I:
        for y in I:
            if x != y:
                counts[(x - y) % c] += 1
    return bool(counts[0] == 0 and np.all(counts[1:] == 1))


def paired_interest_set(I, c):
    """(0, 1, c+1-a_{l-1}, ..., c+1-a_2) for I = (0, 1, a_2, ..., a_{l-1})."""
    I = tuple(I)
    return (0, 1) + tuple(c + 1 - a for a in reversed(I[2:]))


def balanced_chunk_layout(L, c):
    """Reading 1: start/end offsets of c chunks covering range(L)."""
    base, extra = divmod(L, c)
    sizes = [base + (1 if u < extra else 0) for u in range(c)]
    ends = np.cumsum(sizes)
    starts = ends - np.array(sizes)
    return starts.astype(np.int64), ends.astype(np.int64)


def build_tasks(N, c, itr, I):
    """BuildSubseq (Alg. 3) with readings 1-3: every level uses (c, I).

    Returns a list (lexicographic quorum order) of dicts with
      quorum  : tuple (q_1, ..., q_itr)
      tokens  : int64 array of global token ids, ascending
      groups  : list of (bit_index, boolean membership over local tokens)
      bits    : uint32 array, OR of (1 << bit_index) over groups holding the token
    itr = 0 gives the single undecomposed task.
    """
    return build_tasks_levels(N, [(c, tuple(I))] * itr)


def build_tasks_levels(N, levels):
    """BuildSubseq (Alg. 3) with a set per level (reading 5): levels[t] is
    (c_t, I_t) for level t + 1.  Same output as build_tasks."""
    tasks = []
    offsets = np.cumsum([0] + [len(I) - 1 for _, I in levels])
    for quorum in itertools.product(*[range(c) for c, _ in levels]):
        tokens = np.arange(N, dtype=np.int64)
        history = []          # per level: (owner, labels over current tokens)
        for t, q in enumerate(quorum):
            c, I = levels[t]
            L = len(tokens)
            starts, ends = balanced_chunk_layout(L, c)
            labels = np.zeros(L, dtype=np.int64)
            for u in range(c):
                labels[starts[u]:ends[u]] = u
            chunks = sorted(((q + o) % c) for o in I)           # reading 2
            gather = np.concatenate([np.arange(starts[u], ends[u]) for u in chunks])
            history = [(own, lab[gather]) for (own, lab) in history]
            history.append((q, labels[gather]))
            tokens = tokens[gather]
        groups = []
        for t, (owner, labels) in enumerate(history):
            c, I = levels[t]
            for j, o in enumerate(I):
                if j == 0:
                    continue
                chunk = (owner + o) % c
                member = labels == chunk
                groups.append((int(offsets[t]) + (j - 1), member))
        bits = np.zeros(len(tokens), dtype=np.uint32)
        for bit, member in groups:
            bits[member] |= np.uint32(1 << bit)
        tasks.append(dict(quorum=quorum, tokens=tokens, groups=groups, bits=bits))
    return tasks


def local_mask(task, causal):
    """Dense boolean keep-mask of one task (small tasks only)."""
    n = len(task["tokens"])
    keep = np.ones((n, n), dtype=bool)
    for _, member in task["groups"]:
        keep &= ~(member[:, None] & member[None, :])
    if causal:
        g = task["tokens"]
        keep &= g[None, :] <= g[:, None]
    return keep


def coverage_counts(tasks, N, causal):
    """counts[x, y] = number of tasks that hold queries x and keys y and keep
    the pair.  Exactly-once coverage means counts == 1 on every pair dense
    attention keeps (and 0 elsewhere)."""
    counts = np.zeros((N, N), dtype=np.int64)
    for task in tasks:
        g = task["tokens"]
        keep = local_mask(task, causal)
        np.add.at(counts, (g[:, None].repeat(len(g), 1), g[None, :].repeat(len(g), 0)), keep.astype(np.int64))
    return counts


def runs(task):
    """Maximal segments of consecutive global ids with constant bits:
    list of (global_start, length, bits)."""
    g = task["tokens"]; b = task["bits"]
    out = []
    i = 0
    while i < len(g):
        j = i + 1
        while j < len(g) and g[j] == g[j - 1] + 1 and b[j] == b[i]:
            j += 1
        out.append((int(g[i]), int(j - i), int(b[i])))
        i = j
    return out


def block_summaries(bits, block=64):
    """Per `block`-token block: (OR of bits, AND of bits) (App. A.2)."""
    nb = (len(bits) + block - 1) // block
    bor = np.zeros(nb, dtype=np.uint32)
    band = np.zeros(nb, dtype=np.uint32)
    for i in range(nb):
        seg = bits[i * block:(i + 1) * block]
        bor[i] = np.bitwise_or.reduce(seg)
        band[i] = np.bitwise_and.reduce(seg)
    return bor, band


def tile_census(tasks, tile=128, block=64):
    """Pooled census over causal-retained tile x tile regions of every task's
    local score matrix (App. A.2, Fig. "kernel_panels" a).

    A tile (r, s) is causal-retained iff it holds some pair with local key
    index <= local query index, i.e. s <= r.  Each retained tile is classified
    from the block summaries.  Returns (fully_masked, clear, mixed, total)."""
    per = tile // block
    full = clear = mixed = total = 0
    for task in tasks:
        bor, band = block_summaries(task["bits"], block)
        nblk = len(bor)
        ntile = (nblk + per - 1) // per
        tor = np.zeros(ntile, dtype=np.uint32)
        tand = np.full(ntile, 0xFFFFFFFF, dtype=np.uint32)
        for i in range(nblk):
            tor[i // per] |= bor[i]
            tand[i // per] &= band[i]
        r_idx, s_idx = np.tril_indices(ntile)
        is_full = (tand[r_idx] & tand[s_idx]) != 0
        is_clear = (tor[r_idx] & tor[s_idx]) == 0
        full += int(is_full.sum())
        clear += int((is_clear & ~is_full).sum())
        mixed += int((~is_clear & ~is_full).sum())
        total += len(r_idx)
    return full, clear, mixed, total
