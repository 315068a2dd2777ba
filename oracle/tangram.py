"""Plain, slow, fp64 CPU oracle for Tangram's ragged paged attention path.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import or call this module.  It shares no
code with the HIP/C++ library (paper_2606_06302_amd) and never imports it.

Every function restates the method from the paper (Tangram, arXiv 2606.06302)
in the paper's order and notation:

  * retained_lengths  - Budget Reservation, Eq. 4: head (l, h) of a request with
                        context N keeps ceil(B_{l,h} * N) entries.
  * cluster_heads     - Budget-Aware Clustering, Section 4.2.2: sort the heads of
                        each layer by budget, cut into groups of H_p.
  * group_lengths     - Ragged Paging, Section 4.2.1: each group's page table is
                        sized by its longest member.
  * reserve           - Precise Page Allocation, Section 4.1: all pages are
                        reserved once, at admission, from the free list.
  * split_map         - Algorithm 1 (AOT Workload Partitioning).
  * partition_plan    - Algorithm 1's proportional rule applied to one batch's
                        integer retained lengths, then greedy longest-first
                        assignment of the split chunks to persistent workgroups.
  * append_token      - a decode step's new token appended to every head
                        (after its retained entries, within the reservation);
                        partition plans can leave each unit's last chunk open
                        so that one plan serves every later step.
  * decode_attention  - softmax attention of one query token per request over
                        each KV head's retained rows (Eq. 1 with standard
                        scaled-dot-product attention; grouped-query heads share
                        a KV head, Section 2.1).
  * merge_partials    - log-sum-exp merge of split-KV partial results
                        (KV-dimension parallelism, Section 2.2.3).
  * prefill_attention - chunked prefill (Section 2.2.1): a chunk attends to the
                        compressed history of its head and, causally, to itself.
  * prefill_schedule  - ahead-of-time placement of the chunked-prefill
                        workgroups: the same idea as the decode partition
                        (cost known from the retained lengths before the step,
                        Section 4.3), longest-processing-time onto the XCDs.
  * implicit_ratios   - calibration (Section 4.1): the per-head share each head
  * calibrate_budget    gets from the layer-wide top-ceil(rho*H*N) selection
                        (Eq. 3) on a sample, and B = min(1, mu + alpha*sigma)
                        over the samples.
  * release_requests  - request lifecycle: a finished request's pages return to
  * concat_tables       the free list and the surviving tables are compacted;
                        newly admitted requests' tables are appended.
  * memory_footprint  - KV slots each paging scheme allocates for the same
                        retained lengths: the uncompressed cache, a monolithic
                        page table spanning all L x H heads (PagedAttention,
                        Section 4.2.1), and ragged per-group tables.
  * chunk_keep_range  - compression fused into chunked prefill (Section 4.1):
  * top_entries         Eq. 4's per-head Top(ceil(B*N), s) applied to each
  * compress_chunk      chunk as its KV is produced, the kept entries appended
  * compress_plan       to the head's reserved pages, never past the
                        reservation (the overflow rule of Section 4.1).

Readings of points the paper leaves open (each also listed in the design doc):
  - ceil(B*N) is the IEEE fp64 product followed by ceil, with no epsilon.
  - Equal budgets keep ascending head order in the sort (a stable sort).
  - Algorithm 1's round() is round-half-up, floor(x + 0.5), for x >= 0.
  - Pages come off the front of the caller's free list in (request, layer,
    group, page) order; a request that does not fit consumes nothing.
  - A page stores [K|V][slot][token row][head_dim]; slot = a head's position in
    its group.
  - The work unit of the executed partition is (request, KV head); its split
    count follows Algorithm 1's proportional rule on the batch's lengths.
  - Softmax scale 1/sqrt(d) unless given.
  - A prefill chunk sees all of its head's compressed history and, causally
    and inclusively, its own (uncompressed) keys.
  - Eq. 3's global selection ranks like Top() (descending score, NaN last, -0
    equal to +0) with ties broken by the lower flattened index h*N + t.
  - sigma is the population standard deviation over the samples; mu and
    sigma are accumulated in sample order; a budget below `floor` is raised
    to it (the method needs B > 0).
  - Chunk-wise compression keeps, after the first x context tokens, ceil(r*x)
    entries of a head (Eq. 4 on the prefix), capped by the head's reserved
    length; a chunk keeps the difference, so the counts of all chunks of a
    context add up to exactly ceil(r*N).
  - Top() ranks by descending score; equal scores favour the lower token
    index, -0 equals +0, and NaN ranks below every number.  The kept entries
    are stored in ascending token order.
"""
from __future__ import annotations

import heapq
import math

import numpy as np

MODE_AOT, MODE_NAIVE, MODE_UNIFORM, MODE_FILL, MODE_SPLIT_MAP = 0, 1, 2, 3, 4
GROUP_CLUSTERED, GROUP_ADJACENT = 0, 1


class OracleError(ValueError):
    pass


class OutOfPages(OracleError):
    pass


def _check_ratio(r: float):
    if not (r > 0.0 and r <= 1.0):          # also rejects NaN
        raise OracleError(f"budget ratio {r!r} outside (0, 1]")


# ----------------------------------------------------------------- Eq. 4

def retained_lengths(ratio, ctx_len):
    """Eq. 4: every (request b, layer l, KV head h) keeps ceil(r_{b,l,h} * N_b).

    ratio: [B][L][H] float64 in (0, 1]; ctx_len: [B] ints >= 1.
    Returns int64 [B][L][H].
    """
    ratio = np.asarray(ratio, dtype=np.float64)
    Bn, L, H = ratio.shape
    out = np.zeros((Bn, L, H), dtype=np.int64)
    for b in range(Bn):
        n = int(ctx_len[b])
        if n < 1:
            raise OracleError("context length must be >= 1")
        for l in range(L):
            for h in range(H):
                r = float(ratio[b, l, h])
                _check_ratio(r)
                out[b, l, h] = math.ceil(r * n)      # one fp64 multiply, then ceil
    return out


# ------------------------------------------------- Section 4.2.2 clustering

def cluster_heads(budget, heads_per_group, grouping=GROUP_CLUSTERED):
    """Budget-Aware Clustering: pi_l sorts layer l's heads by ascending budget.

    Group i of layer l holds pi_l(j) for j in [i*H_p, (i+1)*H_p).  Returns
    (perm, group_of, slot_of), each int64 [L][H]; slot_of is a head's position
    within its group.  grouping=GROUP_ADJACENT keeps pi_l = identity (the
    paper's "adjacent" alternative in Algorithm 1's comment).
    """
    budget = np.asarray(budget, dtype=np.float64)
    L, H = budget.shape
    if heads_per_group < 1 or H % heads_per_group != 0:
        raise OracleError("H must be a multiple of H_p")
    perm = np.zeros((L, H), dtype=np.int64)
    group_of = np.zeros((L, H), dtype=np.int64)
    slot_of = np.zeros((L, H), dtype=np.int64)
    for l in range(L):
        for h in range(H):
            _check_ratio(float(budget[l, h]))
        if grouping == GROUP_CLUSTERED:
            order = sorted(range(H), key=lambda h: (float(budget[l, h]), h))
        elif grouping == GROUP_ADJACENT:
            order = list(range(H))
        else:
            raise OracleError("unknown grouping")
        for j, h in enumerate(order):
            perm[l, j] = h
            group_of[l, h] = j // heads_per_group
            slot_of[l, h] = j % heads_per_group
    return perm, group_of, slot_of


# ------------------------------------------------- Section 4.2.1 ragged paging

def group_lengths(kv_len, group_of, num_groups):
    """A group's page table holds its longest member: GL = max_{h in g} kv_len."""
    Bn, L, H = kv_len.shape
    gl = np.zeros((Bn, L, num_groups), dtype=np.int64)
    for b in range(Bn):
        for l in range(L):
            for h in range(H):
                g = int(group_of[l, h])
                gl[b, l, g] = max(gl[b, l, g], int(kv_len[b, l, h]))
    return gl


def reserve(ratio, ctx_len, group_of, num_groups, page_size, free_pages, headroom=None):
    """Precise Page Allocation (Section 4.1) into per-group page tables.

    Pages are taken from the front of free_pages in (b, l, g, page) order.  The
    per-(b, l, g) tables are concatenated (the Vectorized Block Table, Section
    4.2.3): table (b, l, g) is pages[offsets[(b*L+l)*G+g] : offsets[...+1]].
    headroom[b] (optional) reserves room for that many decode tokens more in
    every table of request b: each decode step appends one token to every head,
    so every group's length grows by one per step.  Raises OutOfPages,
    consuming nothing, when the list is too short.
    """
    kv_len = retained_lengths(ratio, ctx_len)
    gl = group_lengths(kv_len, group_of, num_groups)
    Bn, L, G = gl.shape
    offsets = np.zeros(Bn * L * G + 1, dtype=np.int64)
    k = 0
    for b in range(Bn):
        extra = 0 if headroom is None else int(headroom[b])
        if extra < 0:
            raise OracleError("negative headroom")
        for l in range(L):
            for g in range(G):
                offsets[(b * L + l) * G + g] = k
                k += -(-(int(gl[b, l, g]) + extra) // page_size)     # ceil((GL + headroom) / P) pages
    offsets[-1] = k
    free_pages = np.asarray(free_pages)
    if k > len(free_pages):
        raise OutOfPages(f"need {k} pages, {len(free_pages)} free")
    pages = free_pages[:k].astype(np.int64).copy()
    return dict(kv_len=kv_len, group_len=gl, offsets=offsets, pages=pages, pages_needed=k)


def memory_footprint(ratio, ctx_len, group_of, num_groups, heads_per_group, page_size):
    """KV slots (one slot = the K and V rows of one token of one head) that each
    paging scheme allocates for the retained lengths of Eq. 4 (Section 4.2.1).

    full:       every request's whole context, paged:  ceil(N/P)*P slots per head.
    retained:   sum of kv_len, what compression keeps.
    monolithic: PagedAttention's single page table spans all L x H heads, so a
                request gets ceil(max_{l,h} kv_len / P) pages for every head.
    ragged:     one table per (request, layer, group) sized by the group's
                longest member: ceil(GL/P) pages of H_p heads.
    Returns a dict of int slot counts plus ragged_pages and page_tables.
    """
    ratio = np.asarray(ratio, dtype=np.float64)
    Bn, L, H = ratio.shape
    P = page_size
    kv_len = retained_lengths(ratio, ctx_len)
    gl = group_lengths(kv_len, group_of, num_groups)
    full = retained = mono = ragged = pages = 0
    for b in range(Bn):
        n = int(ctx_len[b])
        full += -(-n // P) * P * L * H
        longest = 0
        for l in range(L):
            for h in range(H):
                retained += int(kv_len[b, l, h])
                longest = max(longest, int(kv_len[b, l, h]))
            for g in range(num_groups):
                npg = -(-int(gl[b, l, g]) // P)
                pages += npg
                ragged += npg * P * heads_per_group
        mono += -(-longest // P) * P * L * H
    return dict(full_slots=full, retained_slots=retained, monolithic_slots=mono, ragged_slots=ragged,
                ragged_pages=pages, page_tables=Bn * L * num_groups)


def token_location(b, l, h, i, *, num_layers, num_groups, page_size, offsets, pages, group_of, slot_of):
    """Physical (page id, slot, row) of retained entry i of head (b, l, h)."""
    g = int(group_of[l, h])
    table = int(offsets[(b * num_layers + l) * num_groups + g])
    return int(pages[table + i // page_size]), int(slot_of[l, h]), i % page_size


def gather_head(pool, b, l, h, t0, t1, *, geom, offsets, pages, group_of, slot_of):
    """Retained K, V rows t0..t1-1 of head (b, l, h), upcast to fp64.

    pool: [pool_pages][2][H_p][P][d] (any float dtype, numpy).
    """
    d = geom.head_dim
    K = np.zeros((t1 - t0, d), dtype=np.float64)
    V = np.zeros((t1 - t0, d), dtype=np.float64)
    for i in range(t0, t1):
        p, s, r = token_location(b, l, h, i, num_layers=geom.num_layers, num_groups=geom.num_groups,
                                 page_size=geom.page_size, offsets=offsets, pages=pages,
                                 group_of=group_of, slot_of=slot_of)
        K[i - t0] = pool[p, 0, s, r].astype(np.float64)
        V[i - t0] = pool[p, 1, s, r].astype(np.float64)
    return K, V


# ------------------------------------------------------------ Algorithm 1

def _running_sum(values):
    """Left-to-right fp64 sum starting from 0.0 (the order fixes the rounding)."""
    total = 0.0
    for v in values:
        total += float(v)
    return total


def split_map(budget, perm, heads_per_group, n_cta):
    """Algorithm 1 (Section 4.3): a head group gets workgroups in proportion to
    its share of the layer's total budget, and never fewer than one:

        S_{l,i} = max(1, round(Phi_{l,i} / tau_l)),   tau_l = Omega_l / N_CTA,

    Omega_l = the layer's budgets summed over its heads in index order,
    Phi_{l,i} = the budgets of group i (heads perm[l][i*H_p .. (i+1)*H_p - 1])
    summed in that order, all in fp64.  round is half away from zero,
    floor(x + 0.5), not Python's round-half-to-even.  Budgets lie in (0, 1],
    so Omega_l > 0.
    """
    budget = np.asarray(budget, dtype=np.float64)
    L, H = budget.shape
    G = H // heads_per_group
    S = np.zeros((L, G), dtype=np.int64)
    for l in range(L):
        tau = _running_sum(budget[l]) / n_cta
        in_group_order = [budget[l, int(h)] for h in perm[l]]
        for i in range(G):
            phi = _running_sum(in_group_order[i * heads_per_group:(i + 1) * heads_per_group])
            S[l, i] = max(1, math.floor(phi / tau + 0.5))
    return S


# ------------------------------------------- executed partition for one layer

def partition_plan(kv_len, offsets, group_of, slot_of, layer, *, num_layers, num_groups, page_size,
                   mode=MODE_AOT, n_bins=1, split_target=1, bin_weights=None, open_end=False):
    """Balanced split-KV partition of one layer, optionally reusable while the
    lengths grow: with open_end, the chunk that ends a unit (t1 == its length)
    gets t1 = -(capacity of the unit's page table in tokens), meaning "up to
    the head's current length", so the plan stays valid as decode steps append
    tokens (the ahead-of-time plan of Section 4.3 needs no per-step planning).
    """
    plan = _partition_plan(kv_len, offsets, group_of, slot_of, layer, num_layers=num_layers,
                           num_groups=num_groups, page_size=page_size, mode=mode, n_bins=n_bins,
                           split_target=split_target, bin_weights=bin_weights)
    if open_end:
        items = []
        for (pt_base, b, h, slot, t0, t1, out_idx) in plan["items"]:
            if t1 == int(kv_len[b, layer, h]):
                t = (b * num_layers + layer) * num_groups + int(group_of[layer, h])
                t1 = -int(offsets[t + 1] - offsets[t]) * page_size
            items.append((pt_base, b, h, slot, t0, t1, out_idx))
        plan["items"] = items
    return plan


def _partition_plan(kv_len, offsets, group_of, slot_of, layer, *, num_layers, num_groups, page_size,
                    mode=MODE_AOT, n_bins=1, split_target=1, bin_weights=None):
    """Balanced split-KV partition of one layer of one batch.

    Work unit u = (request b, KV head h), in order b, h.  In AOT mode unit u is
    split into s_u = min(ceil(L_u/P), max(1, round_half_up(L_u * T / W)))
    chunks (T = split_target, W = sum of the layer's lengths): Algorithm 1's
    "CTAs proportional to budget share" rule on exact integer lengths.  Chunk c
    covers pages [c*n//s, (c+1)*n//s) of the unit's n = ceil(L_u/P) pages.
    Chunks are then placed longest-first, each on the currently least-loaded of
    n_bins bins (ties: lowest bin).  NAIVE: one chunk per unit, one bin per
    unit.  UNIFORM: every unit gets the same split count ceil(n_bins/units),
    one bin per chunk.

    FILL: the units' pages are laid end to end in (b, h) order and cut into
    n_bins page ranges, one per bin, whose sizes follow bin_weights (all equal
    when None): range k starts at floor(total * (w_0 + ... + w_{k-1}) / sum w).
    A unit is split wherever a range boundary falls inside it, so with equal
    weights every bin gets floor/ceil of total/n_bins pages, and every unit gets
    bins in proportion to its length.

    Returns dict(items=[(pt_base, b, h, slot, t0, t1, out_idx)], bin_offsets,
    unit_splits [B][H], unit_partial_base [B][H], num_partials, bin_load).
    """
    Bn, L, H = kv_len.shape
    P = page_size
    lens = [[int(kv_len[b, layer, h]) for h in range(H)] for b in range(Bn)]
    if mode == MODE_SPLIT_MAP:
        return _split_map_plan(lens, offsets, group_of, slot_of, layer, num_layers, num_groups, P, bin_weights)
    if mode == MODE_FILL:
        return _fill_plan(lens, offsets, group_of, slot_of, layer, num_layers, num_groups, P, n_bins,
                          bin_weights)
    W = sum(sum(r) for r in lens)
    n_units = Bn * H
    splits = np.zeros((Bn, H), dtype=np.int64)
    for b in range(Bn):
        for h in range(H):
            n = -(-lens[b][h] // P)
            if mode == MODE_AOT:
                s = max(1, (2 * lens[b][h] * split_target + W) // (2 * W))
            elif mode == MODE_NAIVE:
                s = 1
            elif mode == MODE_UNIFORM:
                s = max(1, -(-n_bins // n_units))
            else:
                raise OracleError("unknown mode")
            splits[b, h] = min(n, s)
    base = np.full((Bn, H), -1, dtype=np.int64)
    nparts = 0
    for b in range(Bn):
        for h in range(H):
            if splits[b, h] > 1:
                base[b, h] = nparts
                nparts += int(splits[b, h])
    chunks = []          # (t0, t1, b, h, c, item tuple)
    for b in range(Bn):
        for h in range(H):
            n = -(-lens[b][h] // P)
            s = int(splits[b, h])
            g = int(group_of[layer, h])
            pt_base = int(offsets[(b * num_layers + layer) * num_groups + g])
            for c in range(s):
                p0, p1 = c * n // s, (c + 1) * n // s
                t0, t1 = p0 * P, min(p1 * P, lens[b][h])
                out_idx = -1 if s == 1 else int(base[b, h]) + c
                chunks.append((t0, t1, b, h, c, (pt_base, b, h, int(slot_of[layer, h]), t0, t1, out_idx)))
    if mode == MODE_AOT:
        order = sorted(chunks, key=lambda x: (-(x[1] - x[0]), x[2], x[3], x[4]))
        heap = [(0, k) for k in range(n_bins)]
        bins = [[] for _ in range(n_bins)]
        for ch in order:
            load, k = heapq.heappop(heap)
            bins[k].append(ch[5])
            heapq.heappush(heap, (load + (ch[1] - ch[0]), k))
    else:
        # NAIVE: one chunk per unit; UNIFORM: fixed split count.  Either way
        # every chunk is its own bin, in (b, h, c) order.
        bins = [[ch[5]] for ch in chunks]
    items, bin_offsets, bin_load = [], [0], []
    for blist in bins:
        items.extend(blist)
        bin_offsets.append(len(items))
        bin_load.append(sum(it[5] - it[4] for it in blist))
    return dict(items=items, bin_offsets=np.array(bin_offsets, dtype=np.int64),
                unit_splits=splits, unit_partial_base=base, num_partials=nparts,
                bin_load=np.array(bin_load, dtype=np.int64))


def _split_map_plan(lens, offsets, group_of, slot_of, layer, num_layers, num_groups, P, S_row):
    """Algorithm 1's split map used as the executed plan: head group g of this
    layer gets S_row[g] workers, which share the group's work over the whole
    batch (its units (b, h) in (b, h) order, pages laid end to end) in equal
    page ranges.  The groups' bins follow each other in group order."""
    Bn, H = len(lens), len(lens[0])
    pieces = []                               # (bin, (b, h), first page, end page)
    first_bin = 0
    for g in range(num_groups):
        units = [(b, h) for b in range(Bn) for h in range(H) if int(group_of[layer, h]) == g]
        start = [0]
        for b, h in units:
            start.append(start[-1] + -(-lens[b][h] // P))
        total, S = start[-1], int(S_row[g])
        for k in range(S):
            lo, hi = total * k // S, total * (k + 1) // S
            for i, u in enumerate(units):
                a, z = max(lo, start[i]), min(hi, start[i + 1])
                if a < z:
                    pieces.append((first_bin + k, u, a - start[i], z - start[i]))
        first_bin += S
    splits = np.zeros((Bn, H), dtype=np.int64)
    for _, (b, h), _, _ in pieces:
        splits[b, h] += 1
    base = np.full((Bn, H), -1, dtype=np.int64)
    nparts = 0
    for b in range(Bn):
        for h in range(H):
            if splits[b, h] > 1:
                base[b, h] = nparts
                nparts += int(splits[b, h])
    seen = np.zeros((Bn, H), dtype=np.int64)
    bins = [[] for _ in range(first_bin)]
    for k, (b, h), p0, p1 in pieces:
        c = int(seen[b, h])
        seen[b, h] += 1
        pt_base = int(offsets[(b * num_layers + layer) * num_groups + int(group_of[layer, h])])
        out_idx = -1 if splits[b, h] == 1 else int(base[b, h]) + c
        bins[k].append((pt_base, b, h, int(slot_of[layer, h]), p0 * P, min(p1 * P, lens[b][h]), out_idx))
    items, bin_offsets, bin_load = [], [0], []
    for blist in bins:
        items.extend(blist)
        bin_offsets.append(len(items))
        bin_load.append(sum(it[5] - it[4] for it in blist))
    return dict(items=items, bin_offsets=np.array(bin_offsets, dtype=np.int64), unit_splits=splits,
                unit_partial_base=base, num_partials=nparts, bin_load=np.array(bin_load, dtype=np.int64))


def _fill_plan(lens, offsets, group_of, slot_of, layer, num_layers, num_groups, P, n_bins, bin_weights=None):
    Bn, H = len(lens), len(lens[0])
    units = [(b, h) for b in range(Bn) for h in range(H)]
    npages = [-(-lens[b][h] // P) for b, h in units]
    start = [0]
    for n in npages:
        start.append(start[-1] + n)
    total = start[-1]
    weights = [1] * n_bins if bin_weights is None else [int(w) for w in bin_weights]
    before = [0]
    for w in weights:
        before.append(before[-1] + w)
    pieces = []                               # (bin, unit index, first page, end page)
    for k in range(n_bins):
        lo, hi = total * before[k] // before[-1], total * before[k + 1] // before[-1]
        for u in range(len(units)):
            a, z = max(lo, start[u]), min(hi, start[u + 1])
            if a < z:
                pieces.append((k, u, a - start[u], z - start[u]))
    splits = np.zeros((Bn, H), dtype=np.int64)
    for _, u, _, _ in pieces:
        b, h = units[u]
        splits[b, h] += 1
    base = np.full((Bn, H), -1, dtype=np.int64)
    nparts = 0
    for b, h in units:
        if splits[b, h] > 1:
            base[b, h] = nparts
            nparts += int(splits[b, h])
    seen = np.zeros((Bn, H), dtype=np.int64)  # pieces of each unit come in page order
    bins = [[] for _ in range(n_bins)]
    for k, u, p0, p1 in pieces:
        b, h = units[u]
        c = int(seen[b, h])
        seen[b, h] += 1
        pt_base = int(offsets[(b * num_layers + layer) * num_groups + int(group_of[layer, h])])
        out_idx = -1 if splits[b, h] == 1 else int(base[b, h]) + c
        bins[k].append((pt_base, b, h, int(slot_of[layer, h]), p0 * P, min(p1 * P, lens[b][h]), out_idx))
    items, bin_offsets, bin_load = [], [0], []
    for blist in bins:
        items.extend(blist)
        bin_offsets.append(len(items))
        bin_load.append(sum(it[5] - it[4] for it in blist))
    return dict(items=items, bin_offsets=np.array(bin_offsets, dtype=np.int64), unit_splits=splits,
                unit_partial_base=base, num_partials=nparts, bin_load=np.array(bin_load, dtype=np.int64))


# ------------------------------------------------------------- attention

def attend(q_rows, K, V, scale):
    """Softmax attention of query rows [m][d] over keys K [n][d], values V [n][d].

    Returns (O [m][d], lse [m]) in fp64; lse is the natural-log normaliser of
    the scaled logits.
    """
    z = (np.asarray(q_rows, dtype=np.float64) @ K.T) * scale          # [m][n]
    m = z.max(axis=1, keepdims=True)
    w = np.exp(z - m)
    s = w.sum(axis=1, keepdims=True)
    O = (w @ V) / s
    lse = (m + np.log(s))[:, 0]
    return O, lse


def decode_attention(q, pool, layer, *, geom, batch, kv_len, offsets, pages, group_of, slot_of,
                     sm_scale=0.0, heads=None):
    """One decode step of layer `layer`: q [B][Hq][d] -> (O [B][Hq][d], lse [B][Hq]).

    Query head qh reads KV head qh // gqa over its retained kv_len[b, layer, h]
    rows.  `heads` optionally restricts the computation to a list of (b, kv_head)
    pairs (the rest of O stays zero).
    """
    d, gqa = geom.head_dim, geom.gqa
    scale = sm_scale if sm_scale != 0.0 else 1.0 / math.sqrt(d)
    O = np.zeros((batch, geom.num_q_heads, d), dtype=np.float64)
    lse = np.zeros((batch, geom.num_q_heads), dtype=np.float64)
    todo = heads if heads is not None else [(b, h) for b in range(batch) for h in range(geom.num_kv_heads)]
    for b, h in todo:
        n = int(kv_len[b, layer, h])
        K, V = gather_head(pool, b, layer, h, 0, n, geom=geom, offsets=offsets, pages=pages,
                           group_of=group_of, slot_of=slot_of)
        qs = slice(h * gqa, (h + 1) * gqa)
        O[b, qs], lse[b, qs] = attend(q[b, qs], K, V, scale)
    return O, lse


def merge_partials(outs, lses):
    """Log-sum-exp merge: lse* = log sum_i e^{lse_i}; O = sum_i e^{lse_i - lse*} o_i."""
    lses = np.asarray(lses, dtype=np.float64)
    outs = np.asarray(outs, dtype=np.float64)
    m = lses.max(axis=0)
    tot = m + np.log(np.exp(lses - m).sum(axis=0))
    w = np.exp(lses - tot)
    return (w[..., None] * outs).sum(axis=0), tot


def decode_by_plan(q, pool, layer, plan, *, geom, batch, offsets, pages, group_of, slot_of, sm_scale=0.0,
                   live_len=None):
    """Evaluate decode attention chunk by chunk along a partition plan, then merge.

    Split-KV with a log-sum-exp merge is algebraically exact, so this must
    reproduce decode_attention up to fp64 rounding.  An open-ended chunk
    (t1 < 0) runs to the head's current length live_len[b, layer, h], kept
    within [t0 + 1, -t1].
    """
    d, gqa = geom.head_dim, geom.gqa
    scale = sm_scale if sm_scale != 0.0 else 1.0 / math.sqrt(d)
    parts = {}
    for (pt_base, b, h, slot, t0, t1, out_idx) in plan["items"]:
        if t1 < 0:
            t1 = min(max(int(live_len[b, layer, h]), t0 + 1), -t1)
        K, V = gather_head(pool, b, layer, h, t0, t1, geom=geom, offsets=offsets, pages=pages,
                           group_of=group_of, slot_of=slot_of)
        qs = slice(h * gqa, (h + 1) * gqa)
        parts.setdefault((b, h), []).append((t0,) + attend(q[b, qs], K, V, scale))
    O = np.zeros((batch, geom.num_q_heads, d))
    lse = np.zeros((batch, geom.num_q_heads))
    for (b, h), lst in parts.items():
        lst.sort(key=lambda x: x[0])
        qs = slice(h * gqa, (h + 1) * gqa)
        O[b, qs], lse[b, qs] = merge_partials([x[1] for x in lst], [x[2] for x in lst])
    return O, lse


def append_token(k_tok, v_tok, pool, layer, *, geom, live_len, offsets, pages, group_of, slot_of):
    """One decode step's new token, appended to every KV head of one layer.

    k_tok, v_tok [B][H][d]: the token's K and V.  Head (b, layer, h) holding
    n = live_len[b, layer, h] entries stores them as entry n (page layout of
    Section 4.2.1) and then holds n + 1, provided its group's page table has
    room; otherwise nothing is written for that head and it is reported.
    Returns (new pool, new live_len, list of (b, h) that had no room).
    """
    out = pool.copy()
    live = np.array(live_len, dtype=np.int64, copy=True)
    Bn, H = k_tok.shape[0], k_tok.shape[1]
    P, L, G = geom.page_size, geom.num_layers, geom.num_groups
    full = []
    for b in range(Bn):
        for h in range(H):
            n = int(live[b, layer, h])
            t = (b * L + layer) * G + int(group_of[layer, h])
            if n >= int(offsets[t + 1] - offsets[t]) * P:
                full.append((b, h))
                continue
            p, s, r = token_location(b, layer, h, n, num_layers=L, num_groups=G, page_size=P, offsets=offsets,
                                     pages=pages, group_of=group_of, slot_of=slot_of)
            out[p, 0, s, r] = k_tok[b, h]
            out[p, 1, s, r] = v_tok[b, h]
            live[b, layer, h] = n + 1
    return out, live, full


def prefill_attention(q, k_new, v_new, pool, layer, *, geom, kv_len, offsets, pages, group_of, slot_of,
                      sm_scale=0.0, rows=None):
    """Chunked-prefill attention.

    q [B][C][Hq][d]; k_new, v_new [B][C][H][d].  Row i of chunk b for query
    head qh (KV head h = qh // gqa) attends to the kv_len[b, layer, h] retained
    history rows of h followed by chunk keys 0..i.  Returns O [B][C][Hq][d].
    `rows` optionally restricts to a list of (b, qh) pairs.
    """
    Bn, C, Hq, d = q.shape
    gqa = geom.gqa
    scale = sm_scale if sm_scale != 0.0 else 1.0 / math.sqrt(d)
    O = np.zeros((Bn, C, Hq, d), dtype=np.float64)
    todo = rows if rows is not None else [(b, qh) for b in range(Bn) for qh in range(Hq)]
    cache = {}
    for b, qh in todo:
        h = qh // gqa
        if (b, h) not in cache:
            n = int(kv_len[b, layer, h])
            Kh, Vh = gather_head(pool, b, layer, h, 0, n, geom=geom, offsets=offsets, pages=pages,
                                 group_of=group_of, slot_of=slot_of)
            Kc = np.asarray(k_new[b, :, h], dtype=np.float64)
            Vc = np.asarray(v_new[b, :, h], dtype=np.float64)
            cache = {(b, h): (np.concatenate([Kh, Kc]), np.concatenate([Vh, Vc]), n)}
        Kall, Vall, n = cache[(b, h)]
        Q = np.asarray(q[b, :, qh], dtype=np.float64)                   # [C][d]
        z = (Q @ Kall.T) * scale                                         # [C][n + C]
        visible = np.ones_like(z, dtype=bool)
        for i in range(C):
            visible[i, n + i + 1:] = False                               # causal within the chunk
        z = np.where(visible, z, -np.inf)
        m = z.max(axis=1, keepdims=True)
        w = np.exp(z - m)
        O[b, :, qh] = (w @ Vall) / w.sum(axis=1, keepdims=True)
    return O


# ------------------------------------------------------------- prefill schedule

def prefill_schedule(kv_len, layer, chunk_len, gqa, n_xcd, rows_per_block=256, keys_per_tile=64):
    """Workgroup order for chunked prefill, decided ahead of time from the
    retained lengths (the balancing idea of Section 4.3 applied to prefill).

    Block (b, h, rt) covers query rows [rt*rows_per_block, (rt+1)*rows_per_block)
    of unit (b, h), row = i*gqa + j.  It walks ceil(hist/keys_per_tile) history
    tiles and the chunk tiles up to its last chunk row i_last, so its cost is
    ceil(hist/T) + floor(i_last/T) + 1.  Units (all their row tiles together)
    go to XCDs longest first, each to the least-loaded XCD (lowest index on a
    tie); each XCD runs its blocks longest first (ties by unit, then row tile).
    Workgroup k runs on XCD k % n_xcd, so slot k holds the (k // n_xcd)-th block
    of that XCD, coded unit*row_tiles + rt, or -1 past its list.
    """
    kv = np.asarray(kv_len)
    Bn, H = kv.shape[0], kv.shape[2]
    C = chunk_len
    n_rows = C * gqa
    row_tiles = -(-n_rows // rows_per_block)

    def chunk_tiles(rt):
        last_row = min((rt + 1) * rows_per_block, n_rows) - 1
        i_last = min(C - 1, last_row // gqa)
        return i_last // keys_per_tile + 1

    def hist_tiles(u):
        b, h = divmod(u, H)
        return -(-int(kv[b, layer, h]) // keys_per_tile)

    units = list(range(Bn * H))
    cost = {u: sum(hist_tiles(u) + chunk_tiles(rt) for rt in range(row_tiles)) for u in units}
    by_cost = sorted(units, key=lambda u: (-cost[u], u))
    load = [0] * n_xcd
    lists = [[] for _ in range(n_xcd)]
    for u in by_cost:
        x = min(range(n_xcd), key=lambda k: (load[k], k))
        load[x] += cost[u]
        lists[x].extend((u, rt) for rt in range(row_tiles))
    for x in range(n_xcd):
        lists[x].sort(key=lambda ur: (-(hist_tiles(ur[0]) + chunk_tiles(ur[1])), ur[0], ur[1]))
    longest = max(len(v) for v in lists)
    order = []
    for k in range(n_xcd * longest):
        v, j = lists[k % n_xcd], k // n_xcd
        order.append(v[j][0] * row_tiles + v[j][1] if j < len(v) else -1)
    return np.array(order, dtype=np.int64), load


# ------------------------------------ compression fused into chunked prefill

def chunk_keep_range(r, capacity, chunk_start, n_tokens):
    """Entries a prefill chunk keeps for one head (Section 4.1, Eq. 4).

    Once the first x tokens of a context have been compressed, a head with
    ratio r holds ceil(r*x) entries (Eq. 4 applied to the prefix, one fp64
    multiply then ceil), but never more than the `capacity` reserved for it at
    admission: an input that asks for more keeps only its highest-scoring
    entries within the reservation (the overflow rule of Section 4.1).  A chunk
    covering context tokens [c0, c0 + n) finds `cursor` entries already stored
    and keeps `count` more.  Returns (cursor, count).
    """
    _check_ratio(float(r))
    if chunk_start < 0 or n_tokens < 0 or capacity < 0:
        raise OracleError("negative chunk start, token count or capacity")
    cursor = min(math.ceil(float(r) * chunk_start), capacity)
    end = min(math.ceil(float(r) * (chunk_start + n_tokens)), capacity)
    return cursor, end - cursor


def top_entries(scores, k):
    """Top(k, s) of Eq. 4 over one head's chunk: the k highest scores.

    Equal scores favour the lower index, -0.0 equals +0.0 and NaN ranks below
    every number.  Returns the chosen indices in ascending order.
    """
    n = len(scores)
    if not 0 <= k <= n:
        raise OracleError(f"cannot keep {k} of {n} entries")

    def rank_key(t):
        s = float(scores[t])
        return (1, 0.0, t) if math.isnan(s) else (0, -s, t)

    return sorted(sorted(range(n), key=rank_key)[:k])


def compress_chunk(k_new, v_new, scores, pool, layer, *, geom, ratio, capacity, chunk_start, chunk_tokens,
                   offsets, pages, group_of, slot_of):
    """Compress one prefill chunk into the ragged cache (Section 4.1).

    k_new, v_new [B][C][H][d]; scores [B][H][C] (importance of every chunk
    entry, from the compression method's scoring function); ratio [B][L][H];
    capacity [B][L][H] (the reserved retained lengths); chunk_start [B] (context
    tokens before the chunk); chunk_tokens [B] (valid tokens of the chunk).
    For each (b, h) the chunk keeps Top(count, s) of its first chunk_tokens[b]
    entries (chunk_keep_range), written in ascending token order as retained
    entries cursor, cursor+1, ... of the head (page layout of Section 4.2.1).
    Returns (new pool, kept [B][H] lists of chunk indices, cursor [B][H],
    count [B][H]).  `pool` is not modified.
    """
    Bn, C, H, d = k_new.shape
    out = pool.copy()
    cursor = np.zeros((Bn, H), dtype=np.int64)
    count = np.zeros((Bn, H), dtype=np.int64)
    kept = [[None] * H for _ in range(Bn)]
    for b in range(Bn):
        n = int(chunk_tokens[b])
        if not 0 <= n <= C:
            raise OracleError("chunk_tokens outside [0, C]")
        for h in range(H):
            c0, cnt = chunk_keep_range(ratio[b, layer, h], int(capacity[b, layer, h]), int(chunk_start[b]), n)
            idx = top_entries(scores[b, h, :n], cnt)
            for j, t in enumerate(idx):
                p, s, r = token_location(b, layer, h, c0 + j, num_layers=geom.num_layers,
                                         num_groups=geom.num_groups, page_size=geom.page_size, offsets=offsets,
                                         pages=pages, group_of=group_of, slot_of=slot_of)
                out[p, 0, s, r] = k_new[b, t, h]
                out[p, 1, s, r] = v_new[b, t, h]
            cursor[b, h], count[b, h], kept[b][h] = c0, cnt, idx
    return out, kept, cursor, count


def compress_plan(ratio, capacity, chunk_start, chunk_tokens, offsets, group_of, slot_of, layer, *,
                  num_layers, num_groups, rows_per_item):
    """Work items of one chunk's compression: each (b, h) with count > 0, in
    order b, h, is cut into pieces of at most rows_per_item kept entries (by
    rank in ascending token order).  Item = (pt_base, b, h, slot, n_valid,
    cursor, count, rank_begin, rank_end).  Returns (items, cursor, count)."""
    Bn, L, H = np.asarray(ratio).shape
    items = []
    cursor = np.zeros((Bn, H), dtype=np.int64)
    count = np.zeros((Bn, H), dtype=np.int64)
    for b in range(Bn):
        n = int(chunk_tokens[b])
        for h in range(H):
            c0, cnt = chunk_keep_range(ratio[b, layer, h], int(capacity[b, layer, h]), int(chunk_start[b]), n)
            cursor[b, h], count[b, h] = c0, cnt
            base = int(offsets[(b * num_layers + layer) * num_groups + int(group_of[layer, h])])
            for r0 in range(0, cnt, rows_per_item):
                items.append((base, b, h, int(slot_of[layer, h]), n, c0, cnt, r0, min(cnt, r0 + rows_per_item)))
    return items, cursor, count


# ------------------------------------------------ calibration (Section 4.1, Eq. 3)

def implicit_ratios(scores, rho):
    """Implicit per-head retention ratio of one sample under non-uniform
    compression (Eq. 3): per layer, the top ceil(rho*H*N) of the H*N flattened
    scores are kept (descending score, NaN last, -0 equal to +0, ties to the
    lower flattened index h*N + t); head h's ratio is its kept count / N.
    scores [L][H][N]; returns ([L][H] float64 ratios, [L][H] int counts)."""
    scores = np.asarray(scores)
    L, H, N = scores.shape
    if not (0.0 < rho <= 1.0) or N < 1:
        raise OracleError("rho must be in (0, 1] and N >= 1")
    k = math.ceil(float(rho) * (H * N))
    counts = np.zeros((L, H), dtype=np.int64)
    for l in range(L):
        def rank_key(i):
            v = float(scores[l, i // N, i % N])
            return (1, 0.0, i) if math.isnan(v) else (0, -v, i)
        for i in sorted(range(H * N), key=rank_key)[:k]:
            counts[l, i // N] += 1
    ratios = np.zeros((L, H), dtype=np.float64)
    for l in range(L):
        for h in range(H):
            ratios[l, h] = int(counts[l, h]) / N
    return ratios, counts


def calibrate_budget(ratios, alpha, floor):
    """B_{l,h} = min(1, mu + alpha * sigma) over S samples of implicit ratios
    ([S][L][H]), mu the mean and sigma the population standard deviation, both
    accumulated in sample order; raised to `floor` when below it."""
    ratios = np.asarray(ratios, dtype=np.float64)
    S, L, H = ratios.shape
    if S < 1 or not (0.0 < floor <= 1.0) or alpha < 0:
        raise OracleError("need S >= 1, floor in (0, 1], alpha >= 0")
    B = np.zeros((L, H), dtype=np.float64)
    for l in range(L):
        for h in range(H):
            acc = 0.0
            for s_ in range(S):
                acc += float(ratios[s_, l, h])
            mu = acc / S
            var = 0.0
            for s_ in range(S):
                dev = float(ratios[s_, l, h]) - mu
                var += dev * dev
            sigma = math.sqrt(var / S)
            b = mu + float(alpha) * sigma
            B[l, h] = max(float(floor), min(1.0, b))
    return B


# ------------------------------------------------------------ request lifecycle

def release_requests(offsets, pages, finished, num_layers, num_groups):
    """Finished requests give their pages back: returns (freed page ids in table
    order, offsets and pages of the surviving requests' tables, compacted in
    request order; page ids are unchanged)."""
    Bn = len(finished)
    per = num_layers * num_groups
    freed, kept_pages, new_offsets = [], [], []
    for b in range(Bn):
        lo, hi = int(offsets[b * per]), int(offsets[(b + 1) * per])
        if finished[b]:
            freed.extend(int(p) for p in pages[lo:hi])
        else:
            shift = len(kept_pages) - lo
            for t in range(per):
                new_offsets.append(int(offsets[b * per + t]) + shift)
            kept_pages.extend(int(p) for p in pages[lo:hi])
    new_offsets.append(len(kept_pages))
    return np.array(freed, dtype=np.int64), np.array(new_offsets, dtype=np.int64), np.array(kept_pages, dtype=np.int64)


def concat_tables(offsets_a, pages_a, offsets_b, pages_b):
    """The tables of batch b appended after those of batch a (request order a, then b)."""
    n = int(offsets_a[-1])
    offsets = [int(x) for x in offsets_a[:-1]] + [int(x) + n for x in offsets_b]
    return np.array(offsets, dtype=np.int64), np.concatenate([np.asarray(pages_a, dtype=np.int64),
                                                              np.asarray(pages_b, dtype=np.int64)])
