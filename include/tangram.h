/*
 * tangram.h - C ABI of libtangram.so: ragged paged attention over a
 * non-uniformly compressed KV cache on AMD Instinct MI355X (gfx950).
 *
 * The calls follow the problem statement of Tangram (arXiv 2606.06302):
 *   1. per-head budgets fix every head's retained length, and all pages are
 *      reserved once, at admission, in per-group page tables
 *      (Section 4.1 "Budget Reservation", Eq. 4; Section 4.2 "Ragged Paging");
 *   2. heads are clustered by budget into groups of H_p (Section 4.2.2);
 *   3. an ahead-of-time split map / balanced split-KV partition decides how
 *      many workgroups each piece of work gets (Section 4.3, Algorithm 1);
 *   4. ragged paged split-KV decode attention plus a log-sum-exp merge, and a
 *      ragged chunked-prefill attention (Section 2.2, chunked prefill and
 *      KV-dimension parallelism).
 *   5. compression of each prefill chunk into the reserved pages as soon as
 *      its K and V exist (Section 4.1, Eq. 4 per head).
 *
 * Conventions
 *   - Every function returns int32_t: TG_OK (0) or a negative TG_ERR_* code.
 *     tg_last_error() returns a thread-local message describing the most
 *     recent failure on the calling thread.
 *   - The caller owns all memory.  Host calls write only into caller arrays.
 *     Device calls take raw device pointers and a hipStream_t passed as
 *     void*; they enqueue asynchronously, never synchronise, never allocate,
 *     and take any scratch memory from a caller workspace whose size the
 *     matching tg_*_workspace_bytes call reports.
 *   - Arguments are validated on the host before anything is written or
 *     enqueued.  On error nothing is written past what the error's
 *     description says, and no page is consumed.
 *   - Device calls move Q, K, V, tokens, outputs, partials and pool rows with
 *     8- and 16-byte vector accesses: those buffers (and the decode
 *     workspace) must be 16-byte aligned, as hipMalloc's are; a misaligned
 *     one is refused with TG_ERR_INVALID_ARG before anything is enqueued.
 *   - Host integer calls are pure, deterministic and thread-safe (tg_reserve
 *     checks and copies large page lists on up to 16 helper threads, or
 *     TG_HOST_THREADS; results do not depend on the thread count).  The only
 *     library state is a per-device cache of compute-unit counts.
 *   - Physical page layout (Section 4.2.1: a page holds H_p x 2 x P x d
 *     elements for the H_p heads of one group in one layer):
 *         element (page p, kv in {0 = K, 1 = V}, slot s, row t, dim e) at
 *         offset (((p*2 + kv)*H_p + s)*P + t)*d + e   (elements of `dtype`).
 *     Retained entry i of head (b, l, h) lives in page
 *     pt_pages[pt_offsets[(b*L + l)*G + group_of[l][h]] + i / P],
 *     slot slot_of[l][h], row i % P.
 */
#ifndef TANGRAM_H
#define TANGRAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ status codes */
enum {
  TG_OK = 0,
  TG_ERR_INVALID_ARG = -1,     /* malformed argument (bad ratio, shape, id ...) */
  TG_ERR_OUT_OF_PAGES = -2,    /* free list shorter than the reservation needs */
  TG_ERR_BUFFER_TOO_SMALL = -3,/* caller output / workspace buffer too small */
  TG_ERR_UNSUPPORTED = -4,     /* valid but not implemented (head_dim, page size) */
  TG_ERR_HIP = -5,             /* a HIP runtime call or kernel launch failed */
  TG_ERR_NO_MEMORY = -6        /* a host allocation inside a host call failed */
};

/* storage / arithmetic types of Q, K, V and outputs */
enum { TG_F32 = 0, TG_BF16 = 1 };
/* head grouping for tg_cluster_heads */
enum { TG_GROUP_CLUSTERED = 0, TG_GROUP_ADJACENT = 1 };
/* partition modes for tg_build_plan */
enum { TG_PLAN_AOT = 0, TG_PLAN_NAIVE = 1, TG_PLAN_UNIFORM = 2, TG_PLAN_AOT_FILL = 3, TG_PLAN_SPLIT_MAP = 4 };
/* flag OR'ed into a tg_build_plan mode: plans that stay valid while decode
 * steps append tokens (see tg_build_plan) */
enum { TG_PLAN_OPEN_END = 0x100 };

/* Model / cache geometry.  H = num_kv_heads (compression is per KV head,
 * Section 2.1), G = H / heads_per_group groups per layer (must divide),
 * gqa = num_q_heads / num_kv_heads query heads per KV head (must divide);
 * query head qh reads KV head qh / gqa. */
typedef struct {
  int32_t num_layers;      /* L  >= 1 */
  int32_t num_kv_heads;    /* H  >= 1 */
  int32_t num_q_heads;     /* Hq >= H, multiple of H */
  int32_t head_dim;        /* d */
  int32_t page_size;       /* P tokens per page, >= 1 */
  int32_t heads_per_group; /* H_p, divides H */
} tg_geometry;

const char* tg_status_string(int32_t code);   /* static string, never NULL */
const char* tg_last_error(void);              /* thread-local, never NULL */
int32_t     tg_version(void);                 /* (major << 16) | minor */

/* --------------------------------------------- 1a. Budget-Aware Clustering
 * Section 4.2.2.  For each layer l, pi_l is the permutation of the H heads by
 * ascending budget (equal budgets keep ascending head index); group i holds
 * pi_l(j) for j in [i*H_p, (i+1)*H_p).  grouping = TG_GROUP_ADJACENT uses
 * pi_l = identity (the "adjacent" grouping that Algorithm 1 also admits).
 *   budget   [L][H] float64, each in (0, 1]         (host, read)
 *   perm     [L][H] int32 out: perm[l][j] = pi_l(j) (host, written)
 *   group_of [L][H] int32 out: group of head h       (host, written)
 *   slot_of  [L][H] int32 out: position of h in its group, 0..H_p-1
 * Errors: TG_ERR_INVALID_ARG for a NULL pointer, bad geometry, H % H_p != 0,
 * a budget outside (0, 1] or NaN, or an unknown grouping (nothing written). */
int32_t tg_cluster_heads(const tg_geometry* geom, const double* budget, int32_t grouping,
                         int32_t* perm, int32_t* group_of, int32_t* slot_of);

/* ----------------------------- 1b. Budget Reservation + ragged page tables
 * Eq. 4 and Section 4.1 ("Precise Page Allocation"), Section 4.2.1 and 4.2.3.
 *   kv_len[b][l][h]    = ceil(r[b][l][h] * ctx_len[b])   (one fp64 multiply,
 *                        then ceil; r = ratio, or budget broadcast if ratio is NULL)
 *   group_len[b][l][g] = max over heads h of group g of kv_len[b][l][h]
 *   table (b, l, g) holds ceil((group_len + headroom[b])/P) pages: headroom
 *   reserves room for that many decode tokens, which every decode step appends
 *   to every head (tg_append); tables are concatenated in
 *   (b, l, g) order into one CSR array (the Vectorized Block Table):
 *   table (b, l, g) = pt_pages[pt_offsets[(b*L+l)*G+g] .. pt_offsets[...+1]).
 *   Pages are taken from the front of free_pages in that order, so
 *   pt_pages[k] == free_pages[k] for every k < pages_needed.
 * Arguments (all host memory):
 *   batch >= 1; ctx_len [B] int32 >= 1; headroom [B] int32 >= 0, or NULL for none;
 *   ratio [B][L][H] float64 in (0, 1], or NULL to use budget for every request;
 *   budget [L][H] float64 in (0, 1] (read only when ratio is NULL);
 *   group_of [L][H] int32 from tg_cluster_heads;
 *   free_pages [num_free] int32; every id that gets consumed must be in
 *   [0, pool_pages) and distinct;
 *   kv_len [B][L][H] int32 out, group_len [B][L][G] int32 out,
 *   pt_offsets [B*L*G+1] int64 out;
 *   pt_pages [pt_capacity] int32 out, or NULL for a size query;
 *   pages_needed int64 out (always written on TG_OK, and on
 *   TG_ERR_OUT_OF_PAGES / TG_ERR_BUFFER_TOO_SMALL).
 * Returns TG_OK; TG_ERR_OUT_OF_PAGES if num_free < pages_needed (real
 * reservations only: a size query never examines the free list);
 * TG_ERR_BUFFER_TOO_SMALL if pt_pages != NULL and pt_capacity < pages_needed;
 * TG_ERR_INVALID_ARG for bad ratios / lengths / group ids, or consumed page
 * ids that repeat or fall outside the pool.  With pt_pages == NULL the call
 * writes kv_len, group_len, pt_offsets and pages_needed and consumes nothing.
 * On any error pt_pages is left untouched. */
int32_t tg_reserve(const tg_geometry* geom, int32_t batch, const int32_t* ctx_len, const int32_t* headroom,
                   const double* ratio, const double* budget, const int32_t* group_of,
                   const int32_t* free_pages, int64_t num_free, int64_t pool_pages,
                   int32_t* kv_len, int32_t* group_len, int64_t* pt_offsets,
                   int32_t* pt_pages, int64_t pt_capacity, int64_t* pages_needed);

/* ------------------------------------------- 2a. AOT Workload Split Map
 * Algorithm 1, arithmetic in fp64 in the paper's order:
 *   Omega_l = sum_h B[l][h] (h ascending); tau_l = Omega_l / n_cta;
 *   Phi_{l,i} = sum over j in [i*H_p, (i+1)*H_p) of B[l][perm[l][j]];
 *   S[l][i] = max(1, floor(Phi_{l,i} / tau_l + 0.5))   (round half up).
 *   budget [L][H] float64 in (0,1]; perm [L][H] from tg_cluster_heads;
 *   n_cta >= 1; S [L][G] int32 out.  All host memory.
 * Errors: TG_ERR_INVALID_ARG (nothing written). */
int32_t tg_split_map(const tg_geometry* geom, const double* budget, const int32_t* perm,
                     int32_t n_cta, int32_t* S);

/* N_CTA of Section 4.3: the number of decode workgroups the device runs
 * concurrently (HIP occupancy of the decode kernel for this geometry/dtype x
 * compute-unit count of `device`).  n_cta out (host).  Errors:
 * TG_ERR_UNSUPPORTED for shapes the decode kernel does not implement,
 * TG_ERR_HIP if the device query fails. */
int32_t tg_decode_max_ctas(const tg_geometry* geom, int32_t dtype, int32_t device, int32_t* n_cta);

/* ------------------------------- 2b. balanced split-KV partition of a layer
 * Algorithm 1's rule "workgroups proportional to budget share, at least one"
 * applied to this batch's integer retained lengths, with work unit
 * u = (request b, KV head h), units in order b, h.  All arithmetic is int64.
 *   W = sum_u kv_len[b][layer][h];  n_u = ceil(kv_len/P) pages;
 *   AOT:     s_u = min(n_u, max(1, floor((2*kv_len*split_target + W) / (2*W))))
 *   NAIVE:   s_u = 1, and one bin per unit (n_bins ignored: B*H bins)
 *   UNIFORM: s_u = min(n_u, max(1, ceil(n_bins / (B*H)))), one bin per chunk
 *   AOT_FILL: the units' pages laid end to end in unit order are cut into
 *            n_bins ranges [cut_k, cut_{k+1}), cut_k = floor(NP * W_k / W)
 *            (NP = sum n_u, W_k = sum of bin_weights[j] over j < k, W = the
 *            sum of all weights; every weight is 1 when bin_weights is NULL,
 *            giving [k*NP/n_bins, (k+1)*NP/n_bins)); bin k gets the pieces of
 *            the units its range covers (in unit order), so bins hold page
 *            shares in proportion to their weights and every unit gets bins
 *            in proportion to its length; s_u = number of pieces of u.
 *            Weights let a plan give less work to workers that run slower
 *            (e.g. measured per-XCD throughput differences).
 *   SPLIT_MAP: Algorithm 1's split map used as is: bin_weights holds the
 *            layer's row S[layer][0..G-1] of tg_split_map (each in 1..65535;
 *            n_bins is ignored).  Group g's units, in (b, h) order, are laid
 *            end to end and cut like AOT_FILL into S[layer][g] equal page
 *            ranges; the groups' bins follow each other in group order, so
 *            there are sum_g S[layer][g] bins.
 *   chunk c < s_u of unit u covers pages [c*n_u/s_u, (c+1)*n_u/s_u) and tokens
 *   [p0*P, min(p1*P, kv_len)).  out_idx = -1 when s_u == 1, else
 *   unit_partial_base[u] + c (partials numbered over units in order).
 *   AOT bins: chunks sorted by (length desc, b, h, c), each placed on the bin
 *   with the least token load so far (ties: lowest bin), kept in placement
 *   order within a bin.  Items are emitted bin by bin; bin k owns
 *   items[bin_offsets[k] .. bin_offsets[k+1]).
 *   mode | TG_PLAN_OPEN_END: the same plan, except that the chunk that ends a
 *   unit (tok_end == kv_len) gets tok_end = -(capacity of the unit's page
 *   table in tokens).  tg_decode then runs it to the head's live length
 *   (tg_decode_args.live_len), kept within [tok_begin + 1, capacity], so one
 *   plan serves every decode step until the batch changes (Section 4.3: no
 *   planning inside the step).
 * Arguments (host): kv_len [B][L][H] and pt_offsets [B*L*G+1] from tg_reserve;
 *   group_of, slot_of [L][H]; 0 <= layer < L; n_bins >= 1 (AOT, AOT_FILL, UNIFORM);
 *   split_target >= 1 (AOT); bin_weights [n_bins] in 1..65535, or NULL
 *   (AOT_FILL), [G] (SPLIT_MAP, required), NULL otherwise; items [item_capacity] out, or NULL for a size
 *   query (num_items, num_partials and the bin count are still written);
 *   bin_offsets [bins+1] out, where bins = n_bins (AOT, AOT_FILL), B*H (NAIVE), the
 *   number of chunks (UNIFORM) or sum_g S[layer][g] (SPLIT_MAP) - its capacity is
 *   bin_capacity entries;
 *   unit_splits [B][H] out; unit_partial_base [B][H] out (-1 when unsplit);
 *   num_items, num_bins, num_partials out.
 * Errors: TG_ERR_INVALID_ARG; TG_ERR_BUFFER_TOO_SMALL when item_capacity <
 * num_items or bin_capacity < bins + 1 (counts still written). */
typedef struct {
  int64_t pt_base;   /* pt_offsets[(b*L+layer)*G + group_of[layer][h]] */
  int32_t b;         /* request */
  int32_t kv_head;   /* h */
  int32_t slot;      /* slot_of[layer][h] */
  int32_t tok_begin; /* first retained entry, a multiple of P */
  int32_t tok_end;   /* one past the last entry, <= kv_len */
  int32_t out_idx;   /* -1: write the final output; else partial index */
} tg_work_item;      /* 32 bytes */

int32_t tg_build_plan(const tg_geometry* geom, int32_t batch, int32_t layer, const int32_t* kv_len,
                      const int64_t* pt_offsets, const int32_t* group_of, const int32_t* slot_of,
                      int32_t mode, int32_t n_bins, int32_t split_target, const int32_t* bin_weights,
                      tg_work_item* items, int32_t item_capacity,
                      int32_t* bin_offsets, int32_t bin_capacity,
                      int32_t* unit_splits, int32_t* unit_partial_base,
                      int32_t* num_items, int32_t* num_bins, int32_t* num_partials);

/* ------------------------------------ 3. ragged paged decode attention
 * One decode step of one layer (Section 2.2.3 split-KV decoding over the
 * ragged cache of Section 4.2): for every request b and query head qh with
 * KV head h = qh / gqa,
 *   O[b][qh] = softmax(K_h q * sm_scale) V_h   over the retained rows of h,
 * executed as the work items of a tg_build_plan partition: worker k of the
 * decode launch (one wave in the bf16 head_dim-128 kernel, one workgroup
 * otherwise) runs the items of bin k; an item with out_idx >= 0
 * writes an fp32 partial (o, lse) to the workspace, and the partials of every
 * split unit are combined with a log-sum-exp merge: inside the decode launch
 * when merge_counters is given (bf16, head_dim 128), otherwise by a second
 * launch on the same stream (only when num_partials > 0).
 * All pointers below are DEVICE pointers:
 *   q        [B][Hq][d] dtype
 *   kv_pool  [pool_pages][2][H_p][P][d] dtype (layout in the file header);
 *            written only at the rows the append below stores
 *   pt_pages CSR page ids (device copy of tg_reserve's output)
 *   items [num_items], bin_offsets [n_bins+1], unit_splits [B][H],
 *   unit_partial_base [B][H]: device copies of tg_build_plan's output
 *            for the same tables; the kernels read page ids
 *            pt_pages[pt_base + t / P] for t in [tok_begin, tok_end) of
 *            every item without re-checking them against the tables
 *   out      [B][Hq][d] dtype, written for every (b, qh)
 *   lse      [B][Hq] float32 natural-log normaliser, or NULL
 *   workspace >= tg_decode_workspace_bytes(geom, batch, num_partials) bytes
 *            (fp32 partials; no initialisation needed).  Calls that share a
 *            workspace must not overlap in time.
 *   sm_scale: 0 means 1/sqrt(d).
 *   timestamps [n_bins][2] uint64, or NULL: worker k writes the GPU's
 *            constant-rate real-time counter (s_memrealtime, 100 MHz on
 *            MI355X) when it starts bin k and when it has finished it, for
 *            measuring the load imbalance across workers.  Empty bins write
 *            equal stamps.
 *   live_len [B][L][H] int32 or NULL, with layer: current lengths for items
 *            of a TG_PLAN_OPEN_END plan (an open item with live_len NULL runs
 *            to its table's capacity).  Written only by the append below.
 *   merge_counters [B][H] int32 or NULL: arrival counters that let the bf16
 *            head_dim-128 kernel merge split units inside its own launch (the
 *            split piece that finishes last merges its unit), so no second
 *            launch is needed.  They must be zero before the first call; every
 *            call leaves them zero, and calls that share them must not overlap
 *            in time.  NULL, or any other dtype / head_dim: the merge runs as a
 *            second launch on the same stream.  The results are the same
 *            either way, bit for bit.
 *   append_k, append_v [B][H][d] dtype, or both NULL: this step's new token
 *            of every (b, h), appended inside the launch (needs live_len and a
 *            TG_PLAN_OPEN_END plan, whose one open item per unit does it).
 *            The open item of (b, h) reads n = live_len[b][layer][h] and the
 *            capacity cap of its table.  If tok_begin <= n < cap, it attends
 *            over entries [tok_begin, n] with entry n taken from the token
 *            rows, stores those rows as entry n of the cache (the row tg_append
 *            writes) and sets live_len[b][layer][h] to n + 1.  Otherwise it
 *            stores nothing, sets *append_full (when not NULL) to 1 and runs
 *            as without the append.  While every live length is at least the
 *            kv_len the plan was built for (the lengths only grow), one call
 *            gives what tg_append followed by tg_decode gives, bit for bit
 *            (out, lse, cache rows, live_len), in one launch instead of two.
 *   append_full: one int32 the caller clears, or NULL.
 * Supported: dtype TG_F32 or TG_BF16, head_dim 64 or 128, page_size 16,
 * gqa 1..16 (else TG_ERR_UNSUPPORTED).  hip_stream is a hipStream_t (NULL =
 * default stream).  Returns TG_ERR_INVALID_ARG when only one of append_k /
 * append_v is given or the append has no live_len, TG_ERR_HIP if a launch
 * fails. */
typedef struct {
  tg_geometry geom;
  int32_t batch;
  int32_t dtype;
  const void* q;
  void* kv_pool;
  const int32_t* pt_pages;
  const tg_work_item* items;
  const int32_t* bin_offsets;
  int32_t n_bins;
  int32_t num_items;
  const int32_t* unit_splits;
  const int32_t* unit_partial_base;
  int32_t num_partials;
  void* out;
  float* lse;
  float sm_scale;
  void* workspace;
  size_t workspace_bytes;
  uint64_t* timestamps;
  int32_t* live_len;
  int32_t layer;
  int32_t* merge_counters;
  const void* append_k;
  const void* append_v;
  int32_t* append_full;
} tg_decode_args;

size_t  tg_decode_workspace_bytes(const tg_geometry* geom, int32_t batch, int32_t num_partials);
int32_t tg_decode(const tg_decode_args* args, void* hip_stream);

/* 3b. tg_decode without a workspace, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, kernels and results as tg_decode, except
 * that args->workspace and args->workspace_bytes are ignored: the split
 * partials go to a static device array of TG_DECODE_NOALLOC_MAX_BYTES bytes
 * that the library holds on every device it runs on until the process ends.
 * A non-NULL args->merge_counters selects the in-launch merge as in
 * tg_decode, but the counters used are the array's own (its first 64 KiB,
 * for up to 16384 (request, KV head) units; larger batches merge in a second
 * launch), not the pointer passed; the partials get the remaining
 * TG_DECODE_NOALLOC_MAX_BYTES - 64 KiB.
 * The call itself allocates nothing (no hipMalloc, hipFree or allocating
 * library routine); the first call on a device looks up that device's copy
 * of the array (hipGetSymbolAddress), so the device of hip_stream must be the
 * current device.  All calls on one device share the array and it keeps the
 * last call's contents: calls that overlap in time on one device (other
 * streams, other threads) race and must be ordered by the caller.
 * Errors: those of tg_decode; TG_ERR_BUFFER_TOO_SMALL when the plan's
 * partials need more than TG_DECODE_NOALLOC_MAX_BYTES - 64 KiB
 * (tg_decode_workspace_bytes(geom, batch, num_partials) > that; checked
 * on the host, nothing enqueued); TG_ERR_HIP if the lookup fails. */
enum { TG_DECODE_NOALLOC_MAX_BYTES = 16 << 20 };
int32_t tg_decode_noalloc(const tg_decode_args* args, void* hip_stream);

/* 3a. decode-token append (device): one decode step's new token of one layer,
 * written after every KV head's current entries (the cache grows by one token
 * per head per step; Section 2.2, decode, on the ragged layout of Section
 * 4.2).  Head (b, layer, h) with n = live_len[b][layer][h] entries stores the
 * token as entry n (page pt_pages[pt_offsets[t] + n / P], row n % P, t =
 * (b*L + layer)*G + group_of[layer][h]) and live_len becomes n + 1, when its
 * table holds more than n entries; otherwise nothing is written for that head
 * and *full (if not NULL) is set to 1.
 * DEVICE pointers: k_tok, v_tok [B][H][d] dtype; kv_pool; pt_pages,
 * pt_offsets [B*L*G+1]; group_of, slot_of [L][H]; live_len [B][L][H] int32
 * (read and written); full: one int32 the caller clears, or NULL.
 * Supported: dtype TG_F32 or TG_BF16, head_dim 64 or 128.  No workspace. */
typedef struct {
  tg_geometry geom;
  int32_t batch;
  int32_t layer;
  int32_t dtype;
  const void* k_tok;
  const void* v_tok;
  void* kv_pool;
  const int32_t* pt_pages;
  const int64_t* pt_offsets;
  const int32_t* group_of;
  const int32_t* slot_of;
  int32_t* live_len;
  int32_t* full;
} tg_append_args;

int32_t tg_append(const tg_append_args* args, void* hip_stream);

/* ------------------------------- 4. ragged chunked-prefill attention (MFMA)
 * Chunked prefill (Section 2.2.1) over the compressed history (Section 4.1):
 * row i of request b's chunk, query head qh, KV head h = qh / gqa, attends to
 * the kv_len[b][layer][h] retained history rows of h (all visible) followed by
 * chunk keys 0..i (causal, inclusive).  No position encoding is applied
 * (q and k are taken as already rotated).
 * DEVICE pointers:
 *   q     [B][C][Hq][d] bf16      k_new, v_new [B][C][H][d] bf16
 *   kv_pool, pt_pages, pt_offsets [B*L*G+1] int64, kv_len [B][L][H] int32,
 *   group_of, slot_of [L][H] int32   (device copies of the host tables)
 *   out   [B][C][Hq][d] bf16
 *   block_order [num_blocks] int32 from tg_prefill_schedule for the same
 *     geometry, batch, chunk_len, layer and lengths, or NULL: then workgroups
 *     take the (request, KV head) units round-robin over 8 XCDs by index.
 * Work unit: one workgroup per TG_PREFILL_ROWS consecutive query rows
 * (row = i*gqa + j for query head h*gqa + j) of one (b, h); it walks the
 * history and then its causal part of the chunk in tiles of
 * TG_PREFILL_TILE keys.  The result does not depend on block_order.
 * A history length outside [0, pages of the head's table * page_size] is
 * clamped to that range on the device.
 * Supported: dtype TG_BF16, head_dim 64 or 128, page_size 16, gqa 1..16,
 * chunk_len >= 1.  The kernel needs no workspace (workspace may be NULL). */
typedef struct {
  tg_geometry geom;
  int32_t batch;
  int32_t chunk_len;
  int32_t layer;
  int32_t dtype;
  const void* q;
  const void* k_new;
  const void* v_new;
  const void* kv_pool;
  const int32_t* pt_pages;
  const int64_t* pt_offsets;
  const int32_t* kv_len;
  const int32_t* group_of;
  const int32_t* slot_of;
  void* out;
  float sm_scale;
  void* workspace;
  size_t workspace_bytes;
  const int32_t* block_order;
  int32_t num_blocks;
} tg_prefill_args;

enum { TG_PREFILL_ROWS = 256, TG_PREFILL_TILE = 64 };

/* 4a. Ahead-of-time workgroup schedule for tg_prefill (host, integer; the
 * prefill analogue of the balanced decode partition of Section 4.3).
 * The cost of block (b, h, row tile rt) is its tile count
 *   ceil(kv_len[b][layer][h] / TG_PREFILL_TILE) + floor(i_last / TG_PREFILL_TILE) + 1,
 * i_last = min(C-1, (min((rt+1)*TG_PREFILL_ROWS, C*gqa) - 1) / gqa).
 * Units u = b*H + h are placed on n_xcd XCDs longest-processing-time first
 * (descending unit cost, ties by u; each to the least-loaded XCD, ties to the
 * lowest index), so that all row tiles of a unit share one L2; each XCD's
 * blocks run in descending cost (ties by u, rt).  Workgroup k runs on XCD
 * k % n_xcd, so order[k] = the (k / n_xcd)-th block of XCD k % n_xcd,
 * encoded u*row_tiles + rt, or -1 past that XCD's list.
 * Arguments: kv_len [B][L][H] host; n_xcd in 1..64; order [capacity] out or
 * NULL for a size query; num_blocks out (= n_xcd * longest XCD list).
 * Errors: TG_ERR_INVALID_ARG; TG_ERR_BUFFER_TOO_SMALL when capacity <
 * num_blocks (num_blocks still written). */
int32_t tg_prefill_schedule(const tg_geometry* geom, int32_t batch, int32_t chunk_len, int32_t layer,
                            const int32_t* kv_len, int32_t n_xcd, int32_t* order, int32_t capacity,
                            int32_t* num_blocks);

size_t  tg_prefill_workspace_bytes(const tg_prefill_args* args);
int32_t tg_prefill(const tg_prefill_args* args, void* hip_stream);

/* ------------------------- 5. compression fused into chunked prefill
 * Section 4.1 (compression fused into chunked prefill, Eq. 4, overflow
 * handling).  Each prefill chunk is compressed as soon as its K and V exist.
 * For request b and KV head h with selection ratio r = ratio[b][layer][h] (or
 * budget[layer][h] when ratio is NULL) and reserved length
 * cap = kv_len[b][layer][h] (tg_reserve's output for the whole context), a
 * chunk that covers context tokens [c0, c0 + n) (c0 = chunk_start[b],
 * n = chunk_tokens[b]) finds
 *   cursor = min(ceil(r * c0), cap)
 * entries already stored and keeps
 *   count  = min(ceil(r * (c0 + n)), cap) - cursor
 * more (each product one fp64 multiply, then ceil, as in Eq. 4).  Over all
 * chunks of a context the counts add up to ceil(r * N); a selection ratio
 * above the reserved one keeps only the top entries that still fit, the
 * overflow rule.  The kept entries are Top(count) of the chunk's scores:
 * descending score, equal scores favour the lower token index, -0.0 equals
 * +0.0 and NaN ranks below every number.  They are stored in ascending token
 * order as the head's retained entries cursor .. cursor + count - 1 (page
 * layout in the file header).
 *
 * 5a. tg_compress_plan (host, integer): counts and work items of one chunk of
 * one layer.  Units (b, h) with count > 0, in order b, h, are cut into items
 * of at most rows_per_item kept entries, by rank in token order.
 *   chunk_start [B] int32 >= 0; chunk_tokens [B] int32 in [0, chunk_len];
 *   ratio [B][L][H] float64 in (0, 1], or NULL; budget [L][H] float64 (read
 *   when ratio is NULL); kv_len [B][L][H] and pt_offsets from tg_reserve;
 *   group_of, slot_of [L][H]; 0 <= layer < L;
 *   chunk_len in 1..TG_COMPRESS_MAX_CHUNK; rows_per_item in 1..TG_COMPRESS_MAX_ROWS;
 *   items [item_capacity] out, or NULL for a size query;
 *   keep_count [B][H] out (count); write_begin [B][H] out (cursor);
 *   num_items out.  All host memory.
 * Errors: TG_ERR_INVALID_ARG (also when a head's page table holds fewer than
 * kv_len entries, or c0 + n overflows int32); TG_ERR_BUFFER_TOO_SMALL when
 * item_capacity < num_items (keep_count, write_begin and num_items are still
 * written). */
typedef struct {
  int64_t pt_base;    /* pt_offsets[(b*L+layer)*G + group_of[layer][h]] */
  int32_t b;          /* request */
  int32_t kv_head;    /* h */
  int32_t slot;       /* slot_of[layer][h] */
  int32_t n_valid;    /* chunk_tokens[b]: scores past it are not read */
  int32_t cursor;     /* entries of the head stored before this chunk */
  int32_t count;      /* entries this chunk keeps, >= 1 */
  int32_t rank_begin; /* this item writes kept entries [rank_begin, rank_end) */
  int32_t rank_end;
} tg_compress_item;   /* 40 bytes */

enum { TG_COMPRESS_MAX_CHUNK = 16384, TG_COMPRESS_MAX_ROWS = 256, TG_COMPRESS_ONE_LAUNCH_MAX_CHUNK = 1024 };

int32_t tg_compress_plan(const tg_geometry* geom, int32_t batch, int32_t layer, int32_t chunk_len,
                         const int32_t* chunk_start, const int32_t* chunk_tokens, const double* ratio,
                         const double* budget, const int32_t* kv_len, const int64_t* pt_offsets,
                         const int32_t* group_of, const int32_t* slot_of, int32_t rows_per_item,
                         tg_compress_item* items, int32_t item_capacity, int32_t* keep_count,
                         int32_t* write_begin, int32_t* num_items);

/* 5b. tg_compress (device): runs a tg_compress_plan on hip_stream.  For
 * chunk_len > TG_COMPRESS_ONE_LAUNCH_MAX_CHUNK (1024) it takes two launches: the select launch takes one
 * workgroup per (b, h), ranks the chunk's entries and writes the indices of
 * Top(keep_count[b][h]) to kept[]; the copy launch takes one workgroup per
 * item and copies the K and V rows of ranks [rank_begin, rank_end) into their
 * pages.  Shorter chunks take one launch in which every item's wave ranks
 * its unit itself and copies its own ranks.  The results are the same.
 * DEVICE pointers:
 *   k_new, v_new [B][C][H][d] dtype: the chunk's K and V before compression
 *   scores  [B][H][C] float32: importance of every chunk entry (from the
 *           compression method's scoring function); entries at or past
 *           chunk_tokens[b] are ignored (the buffer still holds all C)
 *   kv_pool [pool_pages][2][H_p][P][d] dtype: only the kept rows are written
 *   pt_pages device copy of tg_reserve's output
 *   items [num_items], keep_count [B][H] int32, chunk_tokens [B] int32: device
 *           copies of tg_compress_plan's items and counts and of its input
 *   kept    [B][H][C] int32 (required; it also carries the selection to the
 *           copy launch): kept[(b*H + h)*C + j] = chunk index of the j-th kept
 *           entry in ascending order, for j < keep_count[b][h]; other entries
 *           are left untouched
 * Items and counts must come from one tg_compress_plan call for the same
 * geometry, layer, chunk_len, chunk_tokens and tables; the kernels trust them.
 * Items write disjoint rows; calls that write the same pages or the same kept
 * buffer must be ordered.  Supported: dtype TG_F32 or TG_BF16, head_dim 64 or
 * 128, chunk_len in 1..TG_COMPRESS_MAX_CHUNK (else TG_ERR_UNSUPPORTED /
 * TG_ERR_INVALID_ARG).  No workspace.  num_items == 0 enqueues nothing.
 * Returns TG_ERR_HIP if a launch fails. */
typedef struct {
  tg_geometry geom;
  int32_t batch;
  int32_t chunk_len;
  int32_t dtype;
  const void* k_new;
  const void* v_new;
  const float* scores;
  void* kv_pool;
  const int32_t* pt_pages;
  const tg_compress_item* items;
  int32_t num_items;
  const int32_t* chunk_tokens;
  const int32_t* keep_count;
  int32_t* kept;
} tg_compress_args;

int32_t tg_compress(const tg_compress_args* args, void* hip_stream);

/* ------------------------------------ 6. memory footprint of the paging
 * Section 4.2.1 (a page table spans the heads of one group; PagedAttention is
 * the single group of all L x H heads) and Section 4.2.2.  For the retained
 * lengths kv_len[b][l][h] = ceil(r[b][l][h] * ctx_len[b]) (Eq. 4; r = ratio,
 * or budget broadcast when ratio is NULL), counts KV slots - one slot holds
 * the K and V rows of one token of one head, 2 * d * sizeof(dtype) bytes -
 * that each paging scheme allocates:
 *   full_slots       = sum_b ceil(N_b/P)*P * L*H      (uncompressed, paged)
 *   retained_slots   = sum_{b,l,h} kv_len              (what compression keeps)
 *   monolithic_slots = sum_b ceil(max_{l,h} kv_len/P)*P * L*H
 *                      (one page table spanning every head of the request)
 *   ragged_slots     = sum_{b,l,g} ceil(GL/P)*P * H_p  (one table per group,
 *                      GL = max over the group's heads, groups from group_of)
 *   ragged_pages     = sum_{b,l,g} ceil(GL/P)          (== tg_reserve's count)
 *   page_tables      = B * L * G
 * All host memory; ctx_len [B] >= 1, ratio [B][L][H] or budget [L][H] in
 * (0, 1], group_of [L][H].  Errors: TG_ERR_INVALID_ARG (nothing written). */
typedef struct {
  int64_t full_slots;
  int64_t retained_slots;
  int64_t monolithic_slots;
  int64_t ragged_slots;
  int64_t ragged_pages;
  int64_t page_tables;
} tg_footprint;

int32_t tg_memory_footprint(const tg_geometry* geom, int32_t batch, const int32_t* ctx_len, const double* ratio,
                            const double* budget, const int32_t* group_of, tg_footprint* out);

/* ------------------------------------------------ 7. budget calibration
 * Section 4.1 (budget calibration) and Eq. 3, host, offline.
 * 7a. tg_implicit_ratios: the per-head retention ratio one sample gets under
 * non-uniform compression.  For every layer the top ceil(rho * H * N) of the
 * H*N flattened scores [H][N] are kept (one fp64 multiply, then ceil); the
 * ranking is by descending score, -0.0 equal to +0.0, NaN below every number,
 * ties to the lower flattened index h*N + t.  ratios[l][h] = kept count of
 * head h / N (fp64 division), counts[l][h] the count (or NULL).
 *   scores [L][H][N] float32; rho in (0, 1]; L, H, N >= 1, H*N < 2^31.
 * 7b. tg_calibrate_budget: B[l][h] = min(1, mu + alpha * sigma) over S
 * samples of implicit ratios [S][L][H], mu the mean and sigma the population
 * standard deviation (both summed in sample order, fp64), raised to floor when
 * below it (a head must keep at least some entries).  alpha >= 0, floor in
 * (0, 1].  All host memory.  Errors: TG_ERR_INVALID_ARG (nothing written). */
int32_t tg_implicit_ratios(int32_t num_layers, int32_t num_heads, int32_t n_tokens, const float* scores, double rho,
                           double* ratios, int32_t* counts);
int32_t tg_calibrate_budget(int32_t samples, int32_t num_layers, int32_t num_heads, const double* ratios,
                            double alpha, double floor, double* budget);

/* ------------------------------------------------ 8. request lifecycle
 * Section 4.1 (pages are reserved once at admission) and Section 4.2.3 (the
 * Vectorized Block Table of a batch).  Host, integer.
 * 8a. tg_release_requests: requests with finished[b] != 0 give their pages
 * back: freed receives them in table order (request, layer, group, page);
 * new_offsets / new_pages receive the surviving requests' tables, compacted
 * in request order (page ids unchanged; new_offsets has S*L*G + 1 entries for
 * S survivors).  Pass freed = NULL and new_pages = NULL for a size query
 * (num_freed, num_kept, num_survivors are always written).
 * 8b. tg_concat_tables: the tables of batch b appended after those of batch
 * a: offsets [(Ba+Bb)*L*G + 1], pages [offsets_a[end] + offsets_b[end]].
 * Errors: TG_ERR_INVALID_ARG; TG_ERR_BUFFER_TOO_SMALL when a capacity is short. */
int32_t tg_release_requests(const tg_geometry* geom, int32_t batch, const int64_t* pt_offsets,
                            const int32_t* pt_pages, const uint8_t* finished, int32_t* freed, int64_t freed_capacity,
                            int64_t* new_offsets, int32_t* new_pages, int64_t pages_capacity, int64_t* num_freed,
                            int64_t* num_kept, int32_t* num_survivors);
int32_t tg_concat_tables(const tg_geometry* geom, int32_t batch_a, const int64_t* offsets_a, const int32_t* pages_a,
                         int32_t batch_b, const int64_t* offsets_b, const int32_t* pages_b, int64_t* offsets,
                         int32_t* pages);

/* ------------------------------------- 9. streaming-read ceiling (diagnostic)
 * Measures how fast the device streams the decode kernel's access pattern,
 * so that a decode run can be reported as a fraction of it: for every entry i
 * the K slab and the V slab of (page_ids[i], slots[i]) - P * d elements of
 * dtype each, at the page layout in the file header - are read with 16-byte
 * vector loads, the entries cut into n_workers contiguous ranges (one wave
 * each); worker w stores the XOR of every 32-bit word it read in out[w].
 * DEVICE pointers: kv_pool, page_ids [n], slots [n] (each < H_p), out
 * [n_workers] uint32.  The slab (P * d * sizeof(dtype) bytes) must be 2, 4
 * or 8 KiB (else TG_ERR_UNSUPPORTED, nothing enqueued).  Errors:
 * TG_ERR_INVALID_ARG, TG_ERR_HIP. */
int32_t tg_read_probe(const tg_geometry* geom, int32_t dtype, const void* kv_pool, const int32_t* page_ids,
                      const int32_t* slots, int64_t n, int32_t n_workers, uint32_t* out, void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* TANGRAM_H */
