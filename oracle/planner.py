"""Oracle shard planners (FlashCP Sec. 3.1, 3.3, 3.4; Algorithm 1).

Test infrastructure only (see the package docstring).

A *plan* is an int32 array of shape [m, 4] whose rows are
``(doc, rank, offset, length)``: the ``length`` tokens of document ``doc``
starting ``offset`` tokens into it (the shard's prefix length p_i of
Sec. 3.1) are assigned to CP worker ``rank`` (x_ij = 1). Plans are returned
in canonical form: rows sorted by (doc, offset), empty shards dropped and
adjacent shards of one document on one rank joined (a join changes no
workload, because W is additive over a split of a shard).

Readings of points the paper leaves open (each also listed in the design
notes):

* Per-sequence (the Llama3 CP baseline, Sec. 2.2): as Per-Doc, but the
  whole packed sequence of C tokens is cut at floor(j*C/(2N)), so a chunk
  may span documents (one shard per document it meets).
* Per-Doc (Sec. 2.3): document k of length L is cut at
  ``c_k + floor(j*L/(2N))`` for j = 0..2N; chunk i goes to worker
  ``min(i, 2N-1-i)`` (0-indexed, so worker i gets chunks i and 2N-1-i).
* Least-loaded worker (Algorithm 1, Min_Worker_Add): least workload W,
  ties to the lowest index; documents are sorted by decreasing length,
  ties to the lower document index.
* Max_Token_Worker_Pop / Whole_Doc_Shard_and_Add (Algorithm 1, the
  equal-token loop) are not spelled out. Reading: take the worker with the
  most tokens above C/N (lowest index on ties); pop its whole-document
  pieces last-in-first-out until the popped tokens cover the excess e; the
  worker keeps the tail of the last popped piece so it ends at exactly C/N,
  and gives away that piece's head plus every earlier popped piece. The
  given pieces are handed out in the order they were popped (the head
  last), each from its first token on, to under-full workers, the
  least-loaded (W, then index) first, each taking as many tokens as it has
  room for. Only document prefixes move, matching Sec. 3.3 (only the lower
  segments are exchanged; cost proportional to the moved length).
  If the fullest worker holds no whole-document piece, its excess comes from
  Per-Doc rounding and the loop stops (tokens then differ from C/N by at
  most the number of Per-Doc documents).
* Cur_R (Algorithm 1) is the imbalance of the whole plan, Per-Doc chunks
  included: ``max_j W_j * N / sum_j W_j``, evaluated in IEEE double exactly
  in that order. The loop ends when Cur_R <= R or every document is Per-Doc.

Parity: pinned by closed forms (W, Per-Doc pairs c(2Nc+1)), the
constraints Eq. 1 and Eq. 2, a hand-checked LPT input, brute force over
all whole-document placements for N = 2, and three hybrid inputs worked by
hand under the reading above (two and three workers, up to three passes, a
repair that pops two pieces and splits a given piece over two receivers;
tests/golden/planner_hand.json, tests/test_oracle_planner.py).
"""
from __future__ import annotations

import numpy as np


def shard_work(prefix: int, length: int) -> int:
    """W_i = (2 p_i + s_i + 1) s_i / 2 (Sec. 3.1, Eq. 3): the number of
    (query, key) pairs a shard's queries see under the document mask,
    the diagonal included."""
    return (2 * int(prefix) + int(length) + 1) * int(length) // 2


def _lens(cu) -> list[int]:
    cu = [int(x) for x in cu]
    return [cu[k + 1] - cu[k] for k in range(len(cu) - 1)]


def canonical(rows) -> np.ndarray:
    """Sort by (doc, offset), drop empty shards, join adjacent same-rank ones."""
    rows = sorted((int(d), int(r), int(o), int(l)) for d, r, o, l in rows if int(l) > 0)
    rows.sort(key=lambda t: (t[0], t[2]))
    out: list[list[int]] = []
    for d, r, o, l in rows:
        if out and out[-1][0] == d and out[-1][1] == r and out[-1][2] + out[-1][3] == o:
            out[-1][3] += l
        else:
            out.append([d, r, o, l])
    return np.asarray(out, dtype=np.int32).reshape(-1, 4)


def per_doc_chunks(length: int, cp: int) -> list[tuple[int, int, int]]:
    """Per-Doc sharding of one document (Sec. 2.3): ``(rank, offset, len)``
    of its 2N chunks, chunk i on worker i for i < N and 2N-1-i otherwise."""
    out = []
    for i in range(2 * cp):
        a = (i * length) // (2 * cp)
        b = ((i + 1) * length) // (2 * cp)
        rank = i if i < cp else 2 * cp - 1 - i
        if b > a:
            out.append((rank, a, b - a))
    return out


def plan_per_doc(cu, cp: int) -> np.ndarray:
    """Every document Per-Doc sharded (the Per-Doc CP baseline, Sec. 2.3)."""
    rows = []
    for k, L in enumerate(_lens(cu)):
        rows += [(k, r, o, l) for r, o, l in per_doc_chunks(L, cp)]
    return canonical(rows)


def plan_per_seq(cu, cp: int) -> np.ndarray:
    """The Llama3 CP baseline (Sec. 2.2): the packed sequence of C tokens,
    not each document, is cut into 2N chunks [floor(iC/2N), floor((i+1)C/2N))
    and chunk i goes to worker min(i, 2N-1-i). Written token by token: every
    global position is given its chunk's worker and the runs of equal
    (document, worker) become shards."""
    cu = [int(x) for x in cu]
    total = cu[-1]
    rows = []
    doc = 0
    for g in range(total):
        while g >= cu[doc + 1]:
            doc += 1
        i = (g * 2 * cp) // total
        # g lies in chunk i iff floor(iC/2N) <= g < floor((i+1)C/2N)
        while (i * total) // (2 * cp) > g:
            i -= 1
        while ((i + 1) * total) // (2 * cp) <= g:
            i += 1
        rank = i if i < cp else 2 * cp - 1 - i
        rows.append((doc, rank, g - cu[doc], 1))
    return canonical(rows)


def _sort_order(lens) -> list[int]:
    return sorted(range(len(lens)), key=lambda k: (-lens[k], k))


def _argmin_load(work, allowed=None) -> int:
    best = -1
    for j in range(len(work)):
        if allowed is not None and not allowed[j]:
            continue
        if best < 0 or work[j] < work[best]:
            best = j
    return best


def plan_whole_lpt(cu, cp: int) -> np.ndarray:
    """Whole documents only, each put on the least-loaded worker in order of
    decreasing length (Algorithm 1, the Min_Worker_Add loop). The equal-token
    constraint Eq. 2 is not enforced."""
    lens = _lens(cu)
    work = [0] * cp
    rows = []
    for k in _sort_order(lens):
        j = _argmin_load(work)
        rows.append((k, j, 0, lens[k]))
        work[j] += shard_work(0, lens[k])
    return canonical(rows)


def imbalance(work) -> float:
    """max_j W_j / mean_j W_j (Sec. 3.4), as max*N/sum in IEEE double."""
    s = sum(int(w) for w in work)
    return float(max(int(w) for w in work)) * float(len(work)) / float(s)


def plan_hybrid(cu, cp: int, target_r: float = 1.05):
    """The heuristic of Algorithm 1 under the reading in the module header.

    Returns ``(plan, is_per_doc)`` where ``is_per_doc[k]`` is 1 for documents
    moved to Per-Doc sharding. Requires N | C (Eq. 2's C/N is an integer).
    """
    lens = _lens(cu)
    n = len(lens)
    C = sum(lens)
    if C % cp:
        raise ValueError("context not divisible by CP degree")
    T = C // cp
    order = _sort_order(lens)
    n_per = 0
    while True:
        per_doc, rem = order[:n_per], order[n_per:]
        tokens = [0] * cp
        work = [0] * cp
        fixed = [[] for _ in range(cp)]   # Per-Doc chunks, never popped
        whole = [[] for _ in range(cp)]   # whole-doc pieces, LIFO stacks
        for k in per_doc:
            for r, o, l in per_doc_chunks(lens[k], cp):
                fixed[r].append((k, o, l))
                tokens[r] += l
                work[r] += shard_work(o, l)
        for k in rem:
            j = _argmin_load(work)
            whole[j].append((k, 0, lens[k]))
            tokens[j] += lens[k]
            work[j] += shard_work(0, lens[k])
        # equal-token repair (Eq. 2)
        while any(t != T for t in tokens):
            jstar = max(range(cp), key=lambda j: (tokens[j] - T, -j))
            e = tokens[jstar] - T
            if not whole[jstar]:
                break
            given = []
            got = 0
            while got < e and whole[jstar]:
                piece = whole[jstar].pop()
                given.append(piece)
                got += piece[2]
            if got > e:
                k, o, l = given[-1]
                g = e - (got - l)
                whole[jstar].append((k, o + g, l - g))  # keeps the tail
                given[-1] = (k, o, g)                   # gives the head
            # the donor's tokens and workload, recomputed from what it keeps
            tokens[jstar] = sum(l for _, _, l in fixed[jstar]) + sum(l for _, _, l in whole[jstar])
            work[jstar] = sum(shard_work(o, l) for _, o, l in fixed[jstar]) + \
                sum(shard_work(o, l) for _, o, l in whole[jstar])
            for k, o, l in given:
                pos, left = o, l
                while left > 0:
                    room = [t < T for t in tokens]
                    r = _argmin_load(work, room)
                    take = min(left, T - tokens[r])
                    whole[r].append((k, pos, take))
                    tokens[r] += take
                    work[r] += shard_work(pos, take)
                    pos += take
                    left -= take
        cur_r = imbalance(work)
        if cur_r <= target_r or not rem:
            break
        n_per += 1
    rows = []
    for j in range(cp):
        rows += [(k, j, o, l) for k, o, l in fixed[j]]
        rows += [(k, j, o, l) for k, o, l in whole[j]]
    is_per_doc = np.zeros(n, dtype=np.uint8)
    for k in order[:n_per]:
        is_per_doc[k] = 1
    return canonical(rows), is_per_doc


def validate(cu, cp: int, plan, require_equal_tokens: bool = False) -> None:
    """Raise ValueError unless ``plan`` assigns every token to exactly one
    worker (Eq. 1) and, if asked, every worker holds C/N tokens (Eq. 2)."""
    lens = _lens(cu)
    plan = np.asarray(plan, dtype=np.int64).reshape(-1, 4)
    covered = [np.zeros(L, dtype=np.int64) for L in lens]
    tokens = [0] * cp
    for d, r, o, l in plan:
        if not (0 <= d < len(lens)) or not (0 <= r < cp) or l < 1 or o < 0 or o + l > lens[d]:
            raise ValueError(f"bad shard {(d, r, o, l)}")
        covered[d][o:o + l] += 1
        tokens[r] += l
    for d, c in enumerate(covered):
        if c.size and not (c == 1).all():
            raise ValueError(f"document {d} not covered exactly once")
    if require_equal_tokens:
        C = sum(lens)
        if C % cp or any(t != C // cp for t in tokens):
            raise ValueError("unequal tokens per worker")


def stats(cu, cp: int, plan, hkv: int, d: int) -> dict:
    """Per-worker W, tokens and received-KV tokens; Eq. 4 and Eq. 5 volumes
    (elements, K and V, forward and backward); imbalance ratio."""
    lens = _lens(cu)
    plan = np.asarray(plan, dtype=np.int64).reshape(-1, 4)
    work = [0] * cp
    tokens = [0] * cp
    held = [dict() for _ in range(cp)]   # doc -> (count, last offset + 1)
    last_off = {}
    for dd, r, o, l in plan:
        work[r] += shard_work(o, l)
        tokens[r] += int(l)
        c, hi = held[r].get(int(dd), (0, 0))
        held[r][int(dd)] = (c + int(l), max(hi, int(o + l)))
        last_off[int(dd)] = max(last_off.get(int(dd), -1), int(o))
    recv = [sum(hi - c for c, hi in held[r].values()) for r in range(cp)]
    C = sum(lens)
    eq4 = 4 * C * hkv * d * (cp - 1) // cp
    nonlast = [0] * cp
    for dd, r, o, l in plan:
        if int(o) != last_off[int(dd)]:
            nonlast[r] += int(l)
    eq5 = 4 * max(nonlast) * hkv * d * (cp - 1)
    return dict(work=work, tokens=tokens, recv_tokens=recv, eq4=eq4, eq5=eq5,
                imbalance=imbalance(work))
