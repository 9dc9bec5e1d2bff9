"""Reference sparse index: block-diagonal set, block and column lists, ring shards.

Test infrastructure; see oracle/__init__.py.

Kernel-aware granularity (Section 4.1 (ii)): verticals are kept at token level,
slashes are executed as 64 x 64 tiles of the 64-token grid.  With nb = N / 64
and the selected slash offsets S (delta = n - m):

  * a tile (query block i, key block j) with i - j = Delta holds exactly the
    offsets 64*Delta - 63 .. 64*Delta + 63 (the diagonal tile holds 0..63 once the
    causal mask is applied), so a selected offset delta is covered by the
    block-diagonals {floor(delta/64), ceil(delta/64)}; their union is D
    (entries >= nb have no tile and are dropped);
  * blocks(i) = {i - Delta : Delta in D, Delta <= i}, ascending;
  * cols(i)   = {v in V : v <= 64 i + 63, (i - floor(v/64)) not in D}, ascending:
    the verticals that the selected tiles of row block i do not already cover.

Negative entries of v_idx / s_idx are the unused slots of a top-p list (whose
length varies per head) and are dropped.

Ring shards (Section 4.2 for the striped layout; the zigzag layout is the
baseline the paper compares with): the global 64-token block g belongs to
  striped: worker g mod W;
  zigzag:  chunk c = g // (nb / 2W) belongs to worker c if c < W, else 2W-1-c.
Each worker keeps its own blocks in ascending global order (its local order).
At ring step t, worker r holds the KV shard of worker s = (r - t) mod W; the
step's lists are the whole-sequence lists restricted to the keys of shard s, in
local coordinates (convert_index of Algorithms 1 and 2).

Hierarchical order (Section 4.3, Algorithm 2): the W = nodes x inner workers
run an outer ring over nodes and, inside each outer step, an inner ring over
the node's cards; ring_schedule replays the loops' buffer passing to find which
shard each worker holds at each step.  ring_work and imbalance_degrees give the
worker x shard workload in tile-equivalents and the imbalance degrees of
Section 5's workload balance analysis.
"""
import numpy as np

BLOCK = 64


def diag_set(s_idx, nb: int) -> np.ndarray:
    out = set()
    for delta in np.asarray(s_idx).tolist():
        if delta < 0:          # unused slot
            continue
        for x in (delta // BLOCK, -(-delta // BLOCK)):
            if x < nb:
                out.add(x)
    return np.array(sorted(out), dtype=np.int64)


def owner(g: int, nb: int, W: int, layout: str) -> int:
    if layout == "striped":
        return g % W
    if layout == "zigzag":
        c = g // (nb // (2 * W))
        return c if c < W else 2 * W - 1 - c
    raise ValueError(layout)


def local_blocks(w: int, nb: int, W: int, layout: str) -> np.ndarray:
    return np.array([g for g in range(nb) if owner(g, nb, W, layout) == w], dtype=np.int64)


def ring_schedule(W: int, inner: int = 0) -> np.ndarray:
    """S[r, t] = the worker whose KV shard worker r holds at step t.

    inner = 0 (or 1, or W) is the flat ring: every step each worker passes its
    current KV buffer to worker r + 1.  Otherwise the W workers sit on
    W / inner nodes of `inner` cards (worker r = node * inner + card), and the
    loops of Algorithm 2 are replayed: at the start of each outer step a
    worker posts its current buffer to the same card of the next node; the
    inner loop computes `inner` steps, passing buffers to the next card of the
    same node between them; at the end of the outer step the buffer posted by
    the previous node's card replaces the current one.
    """
    if inner in (0, 1, W):
        inner, nodes = W, 1
        flat = True
    else:
        assert W % inner == 0
        nodes = W // inner
        flat = False
    buf = list(range(W))                     # shard id in each worker's KV buffer
    S = np.zeros((W, W), dtype=np.int64)
    step = 0
    for i in range(nodes):
        posted = list(buf)                   # the outer send takes the buffer as it is now
        for j in range(inner):
            for r in range(W):
                S[r, step] = buf[r]
            step += 1
            if j < inner - 1:                # inner pass: receive from the previous card of the node
                buf = [buf[(r // inner) * inner + (r % inner - 1) % inner] for r in range(W)]
        if i < nodes - 1:                    # outer pass: receive what the previous node posted
            buf = [posted[(r - inner) % W] for r in range(W)]
    if flat:
        assert all(S[r, t] == (r - t) % W for r in range(W) for t in range(W))
    return S


def head_lists(v_idx, s_idx, N: int):
    """Whole-sequence D, blocks(i) and cols(i) for one head."""
    nb = N // BLOCK
    D = diag_set(s_idx, nb)
    in_d = np.zeros(nb, dtype=bool)
    in_d[D] = True
    V = np.unique(np.asarray(v_idx, dtype=np.int64))   # ascending, duplicates count once
    V = V[V >= 0]                                         # unused slots
    blocks, cols = [], []
    for i in range(nb):
        blocks.append(np.sort(i - D[D <= i]))
        cand = V[V <= BLOCK * i + BLOCK - 1]
        cols.append(cand[~in_d[i - cand // BLOCK]])
    return D, blocks, cols


class Index:
    """Index of one ring step (or of the whole sequence when W = 1), all heads.

    Arrays use the library's layout: for flattened head bh = b * Hq + h,
      blk_ptr[bh*nqb + i] .. blk_ptr[bh*nqb + i + 1] bound the ascending local key
      blocks of local query block i in blk_idx; col_ptr / col_idx likewise for
      the local key token offsets of its columns; kblk_ptr / kblk_idx is the
      transpose of the block lists (local query blocks per local key block);
      vcol_ptr[bh] .. vcol_ptr[bh+1] bound the local offsets of the head's
      verticals that this shard owns; diag_bits holds D as a bitset of
      ceil(nb / 32) words per head; q_blk_global / k_blk_global map local blocks
      to global block numbers.
    """

    def __init__(self, v_idx, s_idx, N: int, world: int = 1, rank: int = 0, step: int = 0,
                 layout: str = "striped", inner: int = 0):
        v_idx = np.asarray(v_idx)
        s_idx = np.asarray(s_idx)
        BH = v_idx.shape[0] * v_idx.shape[1]
        v2 = v_idx.reshape(BH, -1)
        s2 = s_idx.reshape(BH, -1)
        nb = N // BLOCK
        W = world
        shard = int(ring_schedule(W, inner)[rank, step]) if W > 1 else 0
        qg = local_blocks(rank, nb, W, layout) if W > 1 else np.arange(nb)
        kg = local_blocks(shard, nb, W, layout) if W > 1 else np.arange(nb)
        kloc = {int(g): j for j, g in enumerate(kg)}
        nqb, nkb = len(qg), len(kg)
        self.N, self.nb, self.nqb, self.nkb, self.BH = N, nb, nqb, nkb, BH
        self.q_blk_global = qg.astype(np.int32)
        self.k_blk_global = kg.astype(np.int32)
        words = (nb + 31) // 32
        self.diag_bits = np.zeros((BH, words), dtype=np.uint32)
        self.blocks = []   # [bh][local qi] -> local key blocks
        self.cols = []     # [bh][local qi] -> local key offsets
        self.vcols = []    # [bh] -> local key offsets of owned verticals
        for bh in range(BH):
            D, blocks, cols = head_lists(v2[bh], s2[bh], N)
            for x in D.tolist():
                self.diag_bits[bh, x // 32] |= np.uint32(1 << (x % 32))
            hb, hc = [], []
            for qi in range(nqb):
                g = int(qg[qi])
                if W == 1:     # whole sequence: local numbering is the global one
                    hb.append(blocks[g])
                    hc.append(cols[g])
                    continue
                hb.append(np.array([kloc[int(j)] for j in blocks[g] if int(j) in kloc], dtype=np.int64))
                hc.append(np.array([kloc[int(c) // BLOCK] * BLOCK + int(c) % BLOCK
                                    for c in cols[g] if int(c) // BLOCK in kloc], dtype=np.int64))
            self.blocks.append(hb)
            self.cols.append(hc)
            V = np.unique(v2[bh].astype(np.int64))
            V = V[V >= 0]
            if W == 1:
                self.vcols.append(V)
                continue
            self.vcols.append(np.array([kloc[int(c) // BLOCK] * BLOCK + int(c) % BLOCK
                                        for c in V if int(c) // BLOCK in kloc], dtype=np.int64))

    # ---- library layout -------------------------------------------------
    def csr(self) -> dict:
        def pack(lists):
            ptr = [0]
            flat = []
            for per_head in lists:
                for ent in per_head:
                    flat.extend(int(x) for x in ent)
                    ptr.append(len(flat))
            return np.array(ptr, dtype=np.int64), np.array(flat, dtype=np.int32)

        kblocks = []
        for bh in range(self.BH):
            per_k = [[] for _ in range(self.nkb)]
            for qi in range(self.nqb):
                for j in self.blocks[bh][qi].tolist():
                    per_k[j].append(qi)
            kblocks.append([np.array(x, dtype=np.int64) for x in per_k])
        blk_ptr, blk_idx = pack(self.blocks)
        col_ptr, col_idx = pack(self.cols)
        kblk_ptr, kblk_idx = pack(kblocks)
        vcol_ptr, vcol_idx = pack([[v] for v in self.vcols])
        return dict(blk_ptr=blk_ptr, blk_idx=blk_idx, col_ptr=col_ptr, col_idx=col_idx,
                    kblk_ptr=kblk_ptr, kblk_idx=kblk_idx, vcol_ptr=vcol_ptr, vcol_idx=vcol_idx,
                    diag_bits=self.diag_bits.reshape(-1).copy(),
                    q_blk_global=self.q_blk_global.copy(), k_blk_global=self.k_blk_global.copy())

    # ---- executed mask --------------------------------------------------
    def mask_rows(self, bh: int, rows) -> np.ndarray:
        """Executed mask for the given local query rows against all local keys.

        M[n, m] is true when m's key block is selected for n's query block or m
        is one of its columns, and the global key position is <= the global
        query position (causal).
        """
        rows = np.asarray(rows, dtype=np.int64)
        nk = self.nkb * BLOCK
        koff = np.arange(nk)
        kpos = self.k_blk_global[koff // BLOCK].astype(np.int64) * BLOCK + koff % BLOCK
        M = np.zeros((len(rows), nk), dtype=bool)
        sel, sel_qi = None, -1
        for r, n in enumerate(rows.tolist()):
            qi = n // BLOCK
            npos = int(self.q_blk_global[qi]) * BLOCK + n % BLOCK
            if qi != sel_qi:           # the keys selected for query block qi (shared by its rows)
                sel = np.zeros(nk, dtype=bool)
                for j in self.blocks[bh][qi].tolist():
                    sel[j * BLOCK:(j + 1) * BLOCK] = True
                sel[self.cols[bh][qi]] = True
                sel_qi = qi
            M[r] = sel & (kpos <= npos)
        return M


def ring_work(v_idx, s_idx, N: int, W: int, layout: str):
    """Selected tiles and column entries of query worker r against KV shard s,
    summed over heads: (tiles[W, W], cols[W, W]), int64.  Worker r computes the
    query blocks it owns; a tile (i, j) or a column c of query block i falls to
    shard owner(j) or owner(c // 64)."""
    v_idx = np.asarray(v_idx)
    s_idx = np.asarray(s_idx)
    BH = v_idx.shape[0] * v_idx.shape[1]
    v2, s2 = v_idx.reshape(BH, -1), s_idx.reshape(BH, -1)
    nb = N // BLOCK
    own = np.array([owner(g, nb, W, layout) for g in range(nb)], dtype=np.int64)
    tiles = np.zeros((W, W), dtype=np.int64)
    cols = np.zeros((W, W), dtype=np.int64)
    for bh in range(BH):
        _, blocks, cl = head_lists(v2[bh], s2[bh], N)
        for i in range(nb):
            np.add.at(tiles[own[i]], own[blocks[i]], 1)
            np.add.at(cols[own[i]], own[cl[i] // BLOCK], 1)
    return tiles, cols


def imbalance_degrees(work, schedule) -> tuple:
    """Imbalance degrees (max / mean) of a worker x shard workload under a step
    schedule S[r, t] (Section 5, workload balance analysis): the worker level
    averages, over steps, max / mean over workers of the step's work; the step
    level averages, over workers, max / mean over that worker's steps."""
    w = np.asarray(work, dtype=np.float64)
    S = np.asarray(schedule)
    W = w.shape[0]
    per_step = np.array([[w[r, S[r, t]] for t in range(W)] for r in range(W)])   # [worker, step]
    worker_level = np.mean([per_step[:, t].max() / per_step[:, t].mean() for t in range(W)])
    step_level = np.mean([per_step[r].max() / per_step[r].mean() for r in range(W)])
    return float(worker_level), float(step_level)
