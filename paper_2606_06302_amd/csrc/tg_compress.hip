// Compression fused into chunked prefill (Tangram, Section 4.1, Eq. 4): the
// per-head Top(count) selection over a chunk's importance scores and the
// scatter of the kept K and V rows into the head's reserved ragged pages.
//
// Chunks of up to kFusedMaxChunk tokens take one launch, one wave per work
// item: the wave ranks its unit's chunk from registers and copies its own
// ranks (tg_compress_wave_kernel).  Longer chunks take two launches on the
// caller's stream:
//   select - one workgroup per (request, KV head) unit, 512 threads up to
//     4096 chunk entries and 1024 above (8 to 16 keys per thread):
//     1. the unit's n scores become order-preserving 32-bit keys in LDS
//        (larger score = larger key; -0 maps to +0; NaN maps to 0, below all);
//     2. a most-significant-digit-first radix select (up to four 8-bit
//        passes, one LDS histogram per wave) finds the count-th largest key T
//        and how many entries equal to T are kept (the lowest-index ones); it
//        stops early once the chosen digit's whole bucket is kept;
//     3. each wave walks its share of the tokens 64 at a time; ballots of
//        the "kept" and "equal to T" predicates and lane-prefix bit counts
//        give every kept entry its rank in token order, written to kept[].
//   copy - one workgroup per work item (at most TG_COMPRESS_MAX_ROWS ranks of
//     one unit): 16-byte loads of the K and V rows named by kept[] from the
//     chunk, 16-byte stores to page pt_pages[pt_base + pos / P], row pos % P,
//     pos = cursor + rank.  These rows are the HBM traffic.
#include <hip/hip_runtime.h>

#include "tg_internal.h"

namespace {

constexpr int kThreads = 256;           // copy launch
constexpr int kBins = 256;              // one radix digit of 8 bits
constexpr int kUnroll = 4;           // rows in flight per thread in the copy launch
constexpr int kBatch = 8;            // score loads / LDS key reads in flight per thread
constexpr int kGroups = 4;           // 64-token groups per batch of the ranking walk
constexpr int kFusedMaxChunk = TG_COMPRESS_ONE_LAUNCH_MAX_CHUNK; // chunks up to this many tokens are compressed in one launch

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

struct SelectParams {
  const uint32_t* scores;            // float32 bit patterns [B][H][C]
  const int32_t* chunk_tokens;       // [B]
  const int32_t* keep_count;         // [B][H]
  int32_t* kept;                     // [B][H][C]
  int32_t H, C;
};

struct CopyParams {
  const u4* k_new;
  const u4* v_new;
  u4* pool;
  const int32_t* pt_pages;
  const tg_compress_item* items;
  const int32_t* kept;
  int32_t H, C, Hp, P;
  int32_t p_shift;                   // log2(P) when P is a power of two, else -1
  int32_t row_u4;                    // 16-byte vectors per K or V row: 8, 16 or 32
};

// Order-preserving key of an fp32 score: a > b as numbers iff key(a) > key(b);
// -0 and +0 share a key; every NaN gets 0, below the key of -inf.
__device__ __forceinline__ uint32_t order_key(uint32_t u) {
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Scalar (constant-cache) loads of values that are uniform across a workgroup.
#define TG_CONST __attribute__((address_space(4)))

__device__ __forceinline__ tg_compress_item load_item(const TG_CONST tg_compress_item* src) {
  tg_compress_item r;
  r.pt_base = src->pt_base;
  r.b = src->b;
  r.kv_head = src->kv_head;
  r.slot = src->slot;
  r.n_valid = src->n_valid;
  r.cursor = src->cursor;
  r.count = src->count;
  r.rank_begin = src->rank_begin;
  r.rank_end = src->rank_end;
  return r;
}

// DPP lane movement with zero fill (row_mask selects the 16-lane rows updated).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_add_src(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, ROW_MASK, 0xF, true);
}

// Inclusive prefix sum over the 64 lanes of a wave: shifts by 1, 2, 4 and 8
// inside each 16-lane row, then row 0's total into row 1 and row 2's into row
// 3 (row_bcast:15), then rows 0-1's total into rows 2 and 3 (row_bcast:31).
__device__ __forceinline__ int wave_inclusive_sum(int x) {
  x += dpp_add_src<0x111, 0xF>(x);
  x += dpp_add_src<0x112, 0xF>(x);
  x += dpp_add_src<0x114, 0xF>(x);
  x += dpp_add_src<0x118, 0xF>(x);
  x += dpp_add_src<0x142, 0xA>(x);
  x += dpp_add_src<0x143, 0xC>(x);
  return x;
}

// Number of set bits of `mask` at lanes below the calling lane.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Top(count) of one unit's chunk scores: the kept chunk indices in ascending
// order go to kept[].  Called by a whole workgroup of kSelThreads threads; keys
// is LDS room for C keys.
template <int kSelThreads>
__device__ __forceinline__ void select_unit(const SelectParams& p, int64_t unit, uint32_t* keys) {
  constexpr int kWaves = kSelThreads / 64;
  // per-wave digit histograms, two buffers: a pass reads one while the
  // waves build the next pass's in the other, each wave clearing its own
  __shared__ __align__(16) uint32_t hist[2][kWaves][kBins];
  __shared__ int32_t wave_cnt[2][kWaves];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = (int)(unit / p.H);
  // the first batch of scores is requested before the counts arrive: it
  // covers chunk entries that exist whatever chunk_tokens says
  const uint32_t* sc = p.scores + unit * p.C;
  uint32_t v[kBatch];
#pragma unroll
  for (int u = 0; u < kBatch; ++u) {
    const int t = tid + u * kSelThreads;
    v[u] = t < p.C ? sc[t] : 0u;
  }
  const int n = min(max(((const TG_CONST int32_t*)p.chunk_tokens)[b], 0), p.C);
  const int count = min(max(((const TG_CONST int32_t*)p.keep_count)[unit], 0), n);
  if (count == 0) return;                        // the whole workgroup leaves together
  const bool keep_all = count >= n;

  if (!keep_all) *reinterpret_cast<u4*>(&hist[0][wave][4 * lane]) = u4(0u);
  // keys into LDS, kBatch loads in flight per thread; the histogram of the
  // top digit is taken on the way
  for (int t0 = tid; t0 < n; t0 += kBatch * kSelThreads) {
    if (t0 != tid) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int t = t0 + u * kSelThreads;
        v[u] = t < n ? sc[t] : 0u;
      }
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int t = t0 + u * kSelThreads;
      if (t < n) {
        const uint32_t key = order_key(v[u]);
        keys[t] = key;
        if (!keep_all) atomicAdd(&hist[0][wave][key >> 24], 1u);
      }
    }
  }
  __syncthreads();   // keys and the first histogram complete

  // radix select over the digits from the top: after each pass, thr holds the
  // digits of the count-th largest key found so far (mask marks them) and
  // need = how many keys with that prefix are kept.  When the whole bucket of
  // the chosen prefix is kept (need == its size), the lower digits cannot
  // change the kept set and the walk stops: the kept keys are then those whose
  // prefix is larger than thr's, or equal to it.  Every wave finds the digit
  // itself, so a pass costs one barrier (after its histogram).
  uint32_t thr = 0, mask = 0;
  int need = count;
  if (!keep_all) {
    int buf = 0;
    for (int shift = 24;; shift -= 8) {
      // lane i owns digits 255-4i .. 252-4i, in descending order
      int c[4] = {0, 0, 0, 0};
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const u4 h = *reinterpret_cast<const u4*>(&hist[buf][w][252 - 4 * lane]);
        c[0] += (int)h.w;
        c[1] += (int)h.z;
        c[2] += (int)h.y;
        c[3] += (int)h.x;
      }
      const int s = c[0] + c[1] + c[2] + c[3];
      int run = wave_inclusive_sum(s) - s;   // matching keys with a larger digit
      int f_digit = -1, f_need = 0, f_whole = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (run < need && run + c[j] >= need) {
          f_digit = 255 - 4 * lane - j;
          f_need = need - run;
          f_whole = run + c[j] == need;       // the bucket is kept whole
        }
        run += c[j];
      }
      // exactly one lane holds the digit: the count-th largest matching key exists
      const uint64_t holder = __ballot(f_digit >= 0);
      const int src = holder ? (int)__builtin_ctzll(holder) : 0;
      const int digit = __builtin_amdgcn_readlane(f_digit, src);
      need = __builtin_amdgcn_readlane(f_need, src);
      thr |= (uint32_t)digit << shift;
      mask |= 0xffu << shift;
      if (__builtin_amdgcn_readlane(f_whole, src) || shift == 0) break;
      // the next digit's histogram over the keys that share the prefix
      buf ^= 1;
      *reinterpret_cast<u4*>(&hist[buf][wave][4 * lane]) = u4(0u);
      for (int t0 = tid; t0 < n; t0 += kBatch * kSelThreads) {
        uint32_t kk[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const int t = t0 + u * kSelThreads;
          kk[u] = t < n ? keys[t] : ~thr;    // ~thr never matches thr under mask (mask != 0 here)
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
          if ((kk[u] & mask) == thr) atomicAdd(&hist[buf][wave][(kk[u] >> (shift - 8)) & 0xffu], 1u);
      }
      __syncthreads();
    }
  }

  // ranks in token order: wave w owns tokens [w*span, (w+1)*span), walked in
  // groups of 64, kGroups groups per batch of LDS reads
  const int span = ((n + kSelThreads - 1) / kSelThreads) * 64;
  const int t_begin = wave * span, t_end = min(n, t_begin + span);
  int gt_w = 0, eq_w = 0;
  for (int base = t_begin; base < t_end; base += 64 * kGroups) {
    uint32_t kk[kGroups];
#pragma unroll
    for (int u = 0; u < kGroups; ++u) {
      const int t = base + 64 * u + lane;
      kk[u] = t < t_end ? keys[t] & mask : 0u;
    }
#pragma unroll
    for (int u = 0; u < kGroups; ++u) {
      const bool valid = base + 64 * u + lane < t_end;
      gt_w += __popcll(__ballot(valid && (keep_all || kk[u] > thr)));
      eq_w += __popcll(__ballot(valid && !keep_all && kk[u] == thr));
    }
  }
  if (lane == 0) {
    wave_cnt[0][wave] = gt_w;
    wave_cnt[1][wave] = eq_w;
  }
  __syncthreads();
  int gt_before = 0, eq_before = 0;
  for (int w = 0; w < wave; ++w) {
    gt_before += wave_cnt[0][w];
    eq_before += wave_cnt[1][w];
  }
  int run_eq = eq_before, run_kept = gt_before + min(eq_before, need);
  int32_t* out = p.kept + unit * p.C;
  for (int base = t_begin; base < t_end; base += 64 * kGroups) {
    uint32_t kk[kGroups];
#pragma unroll
    for (int u = 0; u < kGroups; ++u) {
      const int t = base + 64 * u + lane;
      kk[u] = t < t_end ? keys[t] & mask : 0u;
    }
#pragma unroll
    for (int u = 0; u < kGroups; ++u) {
      const int t = base + 64 * u + lane;
      const bool valid = t < t_end;
      const bool eq = valid && !keep_all && kk[u] == thr;
      const uint64_t eq_mask = __ballot(eq);
      const bool keep = valid && (keep_all || kk[u] > thr || (eq && run_eq + lanes_below(eq_mask) < need));
      const uint64_t keep_mask = __ballot(keep);
      if (keep) out[run_kept + lanes_below(keep_mask)] = t;
      run_eq += __popcll(eq_mask);
      run_kept += __popcll(keep_mask);
    }
  }
}

// kSelThreads: 512 up to 4096 chunk entries, 1024 above (8 to 16 keys per thread)
template <int kSelThreads>
__global__ __launch_bounds__(kSelThreads) void tg_compress_select_kernel(SelectParams p) {
  extern __shared__ uint32_t keys[];             // [C] keys of the unit's scores
  select_unit<kSelThreads>(p, blockIdx.x, keys);
}

// Copies the K and V rows of ranks [r0, r0 + rows) of one unit: rank j's
// chunk index is tok(j); it goes to the head's entry cursor + j.  Called by a
// whole workgroup, kUnroll rows in flight per thread.
template <int kUnroll, typename TokFn>
__device__ __forceinline__ void copy_rows(const CopyParams& p, const tg_compress_item& it, int r0, int rows,
                                          TokFn tok, int tid = threadIdx.x, int nthreads = kThreads) {
  const int lpr = p.row_u4;
  const int rpp = nthreads / lpr;               // rows per pass of the thread group
  const int sub = tid % lpr, rsel = tid / lpr;
  const int64_t tok_stride = (int64_t)p.H * lpr;
  const int64_t src0 = ((int64_t)it.b * p.C * p.H + it.kv_head) * lpr + sub;
  const int64_t v_plane = (int64_t)p.Hp * p.P * lpr;  // V rows of a page follow its K rows
  for (int base = 0; base < rows; base += kUnroll * rpp) {
    // every load of the batch (K row, V row, destination page id) goes out
    // before the first result is used, so a batch costs one memory round trip
    // (straight-line: rows past the end load the last row again and store nothing)
    u4 kk[kUnroll], vv[kUnroll];
    int32_t page[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int j = min(base + u * rpp + rsel, rows - 1);
      const int t = min(max(tok(j), 0), p.C - 1);   // in range by construction; clamped for safety
      const int64_t src = src0 + t * tok_stride;
      kk[u] = p.k_new[src];
      vv[u] = p.v_new[src];
      const int pos = it.cursor + r0 + j;
      page[u] = p.pt_pages[it.pt_base + (p.p_shift >= 0 ? pos >> p.p_shift : pos / p.P)];
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int j = base + u * rpp + rsel;
      if (j < rows) {
        const int pos = it.cursor + r0 + j;
        const int row = p.p_shift >= 0 ? pos & (p.P - 1) : pos % p.P;
        const int64_t dst = (((int64_t)page[u] * 2 * p.Hp + it.slot) * p.P + row) * lpr + sub;
        p.pool[dst] = kk[u];
        p.pool[dst + v_plane] = vv[u];
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void tg_compress_copy_kernel(CopyParams p) {
  const tg_compress_item it = load_item((const TG_CONST tg_compress_item*)p.items + blockIdx.x);
  const int r0 = max(it.rank_begin, 0);
  const int r1 = min(min(it.rank_end, min(it.count, p.C)), r0 + TG_COMPRESS_MAX_ROWS);
  const int32_t* src_tok = p.kept + ((int64_t)it.b * p.H + it.kv_head) * p.C + r0;
  copy_rows<kUnroll>(p, it, r0, r1 - r0, [&](int j) { return src_tok[j]; });
}

// Short chunks in one launch, one single-wave workgroup per work item and no
// barrier: the wave holds its unit's whole chunk of keys in registers (lane
// l, slot i: token 64*i + l, so the score loads are coalesced and token order
// is slot-major), finds the count-th largest key with the same
// most-significant-digit radix select as select_unit (the digit histogram in
// the wave's LDS, whose operations a wave executes in order), ranks the kept
// entries by ballots in token order, and copies its own ranks.  The unit's
// first item also writes kept[].  KPL = keys per lane.  Single-wave
// workgroups spread the items over every CU (measured at chunk 512: 7.9 us,
// against 8.1, 9.3 and 12.1 us with 4, 8 and 16 items per workgroup).
template <int KPL>
__global__ __launch_bounds__(64) void tg_compress_wave_kernel(SelectParams sp, CopyParams p, int32_t n_items) {
  constexpr int kSpill = kFusedMaxChunk;        // per-lane dummy entries for branch-free stores
  __shared__ __align__(16) uint32_t hist[kBins];
  __shared__ int32_t kept_lds[kFusedMaxChunk + 64];
  const int lane = threadIdx.x;
  const int item = blockIdx.x;
  if (item >= n_items) return;
  const tg_compress_item it = load_item((const TG_CONST tg_compress_item*)p.items + item);
  const int64_t unit = (int64_t)it.b * p.H + it.kv_head;
  const int C = sp.C;
  // every score load goes out before the counts arrive: entries below C exist whatever chunk_tokens says
  const uint32_t* sc = sp.scores + unit * C;
  uint32_t key[KPL];
#pragma unroll
  for (int i = 0; i < KPL; ++i) {
    const int t = 64 * i + lane;
    key[i] = t < C ? sc[t] : 0u;
  }
  const int n = min(max(((const TG_CONST int32_t*)sp.chunk_tokens)[it.b], 0), C);
  const int count = min(max(((const TG_CONST int32_t*)sp.keep_count)[unit], 0), n);
  if (count == 0) return;
  const bool keep_all = count >= n;
#pragma unroll
  for (int i = 0; i < KPL; ++i) key[i] = order_key(key[i]);

  // after the select, the kept keys are those whose prefix (mask) is above
  // thr, and `need` of those whose prefix equals thr (the lowest-index ones);
  // whole: every key with prefix thr is kept
  uint32_t thr = 0, mask = 0;
  int need = count;
  bool whole = true;
  if (!keep_all) {
    for (int shift = 24;; shift -= 8) {
      *reinterpret_cast<u4*>(&hist[4 * lane]) = u4(0u);
#pragma unroll
      for (int i = 0; i < KPL; ++i)
        if (64 * i + lane < n && (key[i] & mask) == thr) atomicAdd(&hist[(key[i] >> shift) & 0xffu], 1u);
      // lane i owns digits 255-4i .. 252-4i, in descending order
      const u4 hv = *reinterpret_cast<const u4*>(&hist[252 - 4 * lane]);
      const int c[4] = {(int)hv.w, (int)hv.z, (int)hv.y, (int)hv.x};
      const int s = c[0] + c[1] + c[2] + c[3];
      int run = wave_inclusive_sum(s) - s;   // matching keys with a larger digit
      int f_digit = -1, f_need = 0, f_whole = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (run < need && run + c[j] >= need) {
          f_digit = 255 - 4 * lane - j;
          f_need = need - run;
          f_whole = run + c[j] == need;
        }
        run += c[j];
      }
      const uint64_t holder = __ballot(f_digit >= 0);
      const int src = holder ? (int)__builtin_ctzll(holder) : 0;
      const int digit = __builtin_amdgcn_readlane(f_digit, src);
      need = __builtin_amdgcn_readlane(f_need, src);
      whole = __builtin_amdgcn_readlane(f_whole, src) != 0;
      thr |= (uint32_t)digit << shift;
      mask |= 0xffu << shift;
      if (whole || shift == 0) break;
    }
  }

  // ranks in token order (slot-major); a lane that keeps nothing in a slot
  // stores to its own dummy entry instead of branching
  int32_t* kl = kept_lds;
  int run_eq = 0, run_kept = 0;
#pragma unroll
  for (int i = 0; i < KPL; ++i) {
    const int t = 64 * i + lane;
    const bool valid = t < n;
    const uint32_t kk = key[i] & mask;
    bool keep;
    if (keep_all) {
      keep = valid;
    } else if (whole) {
      keep = valid && kk >= thr;
    } else {   // only the lowest-index `need` keys equal to thr are kept
      const bool eq = valid && kk == thr;
      const uint64_t eq_mask = __ballot(eq);
      keep = valid && (kk > thr || (eq && run_eq + lanes_below(eq_mask) < need));
      run_eq += __popcll(eq_mask);
    }
    const uint64_t keep_mask = __ballot(keep);
    kl[keep ? run_kept + lanes_below(keep_mask) : kSpill + lane] = t;
    run_kept += __popcll(keep_mask);
  }
  const int r0 = max(it.rank_begin, 0);
  const int r1 = min(min(it.rank_end, min(count, min(it.count, p.C))), r0 + TG_COMPRESS_MAX_ROWS);
  copy_rows<8>(p, it, r0, r1 - r0, [&](int j) { return kl[r0 + j]; }, lane, 64);
  if (it.rank_begin == 0) {
    int32_t* out = sp.kept + unit * p.C;
    for (int r = lane; r < count; r += 64) out[r] = kl[r];
  }
}

}  // namespace

extern "C" int32_t tg_compress(const tg_compress_args* a, void* hip_stream) {
  if (!a) return tg::fail(TG_ERR_INVALID_ARG, "args is NULL");
  const tg_geometry& g = a->geom;
  if (int32_t rc = tg::check_geometry(&g)) return rc;
  if (a->dtype != TG_F32 && a->dtype != TG_BF16) return tg::fail(TG_ERR_UNSUPPORTED, "dtype must be f32 or bf16");
  if (g.head_dim != 64 && g.head_dim != 128)
    return tg::fail(TG_ERR_UNSUPPORTED, "compression supports head_dim 64 or 128 (got %d)", g.head_dim);
  if (a->batch < 1) return tg::fail(TG_ERR_INVALID_ARG, "batch must be >= 1");
  if (a->chunk_len < 1 || a->chunk_len > TG_COMPRESS_MAX_CHUNK)
    return tg::fail(TG_ERR_INVALID_ARG, "chunk_len %d outside [1, %d]", a->chunk_len, (int)TG_COMPRESS_MAX_CHUNK);
  if (a->num_items < 0) return tg::fail(TG_ERR_INVALID_ARG, "num_items < 0");
  if (a->num_items == 0) return TG_OK;
  if (!a->k_new || !a->v_new || !a->scores || !a->kv_pool || !a->pt_pages || !a->items || !a->chunk_tokens ||
      !a->keep_count || !a->kept)
    return tg::fail(TG_ERR_INVALID_ARG, "NULL device pointer");
  if (!tg::aligned16({a->k_new, a->v_new, a->kv_pool}))
    return tg::fail(TG_ERR_INVALID_ARG, "device buffers must be 16-byte aligned");
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  SelectParams s;
  CopyParams c;
  c.k_new = static_cast<const u4*>(a->k_new);
  c.v_new = static_cast<const u4*>(a->v_new);
  c.pool = static_cast<u4*>(a->kv_pool);
  c.pt_pages = a->pt_pages;
  c.items = a->items;
  c.kept = a->kept;
  c.H = g.num_kv_heads;
  c.C = a->chunk_len;
  c.Hp = g.heads_per_group;
  c.P = g.page_size;
  c.p_shift = (g.page_size & (g.page_size - 1)) == 0 ? __builtin_ctz((unsigned)g.page_size) : -1;
  c.row_u4 = g.head_dim * (a->dtype == TG_F32 ? 4 : 2) / 16;
  s.scores = reinterpret_cast<const uint32_t*>(a->scores);
  s.chunk_tokens = a->chunk_tokens;
  s.keep_count = a->keep_count;
  s.kept = a->kept;
  s.H = g.num_kv_heads;
  s.C = a->chunk_len;
  if (a->chunk_len <= kFusedMaxChunk) {
    const int kpl = (a->chunk_len + 63) / 64;
    const dim3 grid((unsigned)a->num_items), block(64);
    if (kpl <= 1) hipLaunchKernelGGL(tg_compress_wave_kernel<1>, grid, block, 0, stream, s, c, a->num_items);
    else if (kpl <= 2) hipLaunchKernelGGL(tg_compress_wave_kernel<2>, grid, block, 0, stream, s, c, a->num_items);
    else if (kpl <= 4) hipLaunchKernelGGL(tg_compress_wave_kernel<4>, grid, block, 0, stream, s, c, a->num_items);
    else if (kpl <= 8) hipLaunchKernelGGL(tg_compress_wave_kernel<8>, grid, block, 0, stream, s, c, a->num_items);
    else hipLaunchKernelGGL(tg_compress_wave_kernel<16>, grid, block, 0, stream, s, c, a->num_items);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "compress launch failed: %s", hipGetErrorString(e));
    return TG_OK;
  }
  const size_t lds = (size_t)a->chunk_len * sizeof(uint32_t);
  const bool wide = a->chunk_len > 4096;
  const void* select = wide ? reinterpret_cast<const void*>(tg_compress_select_kernel<1024>)
                            : reinterpret_cast<const void*>(tg_compress_select_kernel<512>);
  if (lds > 32768) {
    hipError_t e = hipFuncSetAttribute(select, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "compress LDS attribute: %s", hipGetErrorString(e));
  }
  if (wide)
    hipLaunchKernelGGL(tg_compress_select_kernel<1024>, dim3(a->batch * g.num_kv_heads), dim3(1024), lds, stream, s);
  else
    hipLaunchKernelGGL(tg_compress_select_kernel<512>, dim3(a->batch * g.num_kv_heads), dim3(512), lds, stream, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "compress select launch failed: %s", hipGetErrorString(e));
  hipLaunchKernelGGL(tg_compress_copy_kernel, dim3(a->num_items), dim3(kThreads), 0, stream, c);
  e = hipGetLastError();
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "compress copy launch failed: %s", hipGetErrorString(e));
  return TG_OK;
}
