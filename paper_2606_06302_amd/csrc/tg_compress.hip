// Compression fused into chunked prefill (Tangram, Section 4.1, Eq. 4): the
// per-head Top(count) selection over a chunk's importance scores and the
// scatter of the kept K and V rows into the head's reserved ragged pages.
//
// One workgroup of 256 threads per work item (at most TG_COMPRESS_MAX_ROWS
// kept entries of one (request, KV head) unit):
//   1. the unit's n scores become order-preserving 32-bit keys in LDS
//      (larger score = larger key; -0 maps to +0; NaN maps to 0, below all);
//   2. a most-significant-digit-first radix select (four 8-bit passes over
//      LDS histograms) finds the count-th largest key T and how many entries
//      equal to T are kept (the lowest-index ones);
//   3. two workgroup prefix sums over contiguous token runs give every kept
//      entry its rank in token order;
//   4. the item's ranks are copied row by row with 16-byte loads from the
//      chunk's K and V and 16-byte stores into page pt_pages[pt_base + pos/P],
//      row pos % P, pos = cursor + rank.
// Every item of a unit repeats the selection (it reads n scores, a few KB
// from L2); the K/V rows are the HBM traffic, each read and written once.
#include <hip/hip_runtime.h>

#include "tg_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kBins = 256;           // one radix digit of 8 bits; == kThreads
constexpr int kUnroll = 4;           // rows in flight per thread in the copy

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

struct CompressParams {
  const u4* k_new;
  const u4* v_new;
  const uint32_t* scores;            // float32 bit patterns
  u4* pool;
  const int32_t* pt_pages;
  const tg_compress_item* items;
  int32_t* kept;
  int32_t H, C, Hp, P;
  int32_t row_u4;                    // 16-byte vectors per K or V row: 8, 16 or 32
};

// Order-preserving key of an fp32 score: a > b as numbers iff key(a) > key(b);
// -0 and +0 share a key; every NaN gets 0, below the key of -inf.
__device__ __forceinline__ uint32_t order_key(uint32_t u) {
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int wave_inclusive_sum(int x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

// Exclusive prefix sum over the workgroup in thread order; *total gets the sum.
__device__ __forceinline__ int block_exclusive_sum(int v, int* wave_tot, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int inc = wave_inclusive_sum(v, lane);
  if (lane == 63) wave_tot[wave] = inc;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int t = wave_tot[w];
    before += (w < wave) ? t : 0;
    all += t;
  }
  __syncthreads();  // wave_tot is reused by the next sum
  *total = all;
  return before + inc - v;
}

__global__ __launch_bounds__(kThreads) void tg_compress_kernel(CompressParams p) {
  extern __shared__ uint32_t keys[];             // [n] keys of the unit's scores
  __shared__ uint32_t hist[kBins];
  __shared__ int32_t rows_src[TG_COMPRESS_MAX_ROWS];  // chunk index of each rank of the item
  __shared__ int32_t wave_tot[kWaves];
  __shared__ uint32_t pick[2];

  const tg_compress_item it = p.items[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // the plan guarantees these bounds; clamping keeps a malformed item inside its buffers
  const int n = min(max(it.n_valid, 0), p.C);
  const int count = min(max(it.count, 0), n);
  const int r0 = max(it.rank_begin, 0);
  const int r1 = min(min(it.rank_end, count), r0 + TG_COMPRESS_MAX_ROWS);
  const int64_t unit = (int64_t)it.b * p.H + it.kv_head;

  const uint32_t* sc = p.scores + unit * p.C;
  for (int t = tid; t < n; t += kThreads) keys[t] = order_key(sc[t]);
  __syncthreads();

  // 1-2. radix select: thr = the count-th largest key, need = entries equal to
  // thr that are kept
  const bool keep_all = count >= n;
  uint32_t thr = 0, mask = 0;
  int need = count;
  if (!keep_all) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      hist[tid] = 0;
      __syncthreads();
      for (int t = tid; t < n; t += kThreads) {
        const uint32_t key = keys[t];
        if ((key & mask) == thr) atomicAdd(&hist[(key >> shift) & 0xffu], 1u);
      }
      __syncthreads();
      if (wave == 0) {
        // lane i owns digits 255-4i .. 252-4i, in descending order
        int c[4], s = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          c[j] = (int)hist[255 - 4 * lane - j];
          s += c[j];
        }
        int run = wave_inclusive_sum(s, lane) - s;  // matching keys with a larger digit
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (run < need && run + c[j] >= need) {
            pick[0] = 255u - 4u * lane - j;
            pick[1] = (uint32_t)(need - run);
          }
          run += c[j];
        }
      }
      __syncthreads();
      thr |= pick[0] << shift;
      mask |= 0xffu << shift;
      need = (int)pick[1];
    }
  }

  // 3. ranks in token order over contiguous runs of m tokens per thread
  const int m = (n + kThreads - 1) / kThreads;
  const int a = min(n, tid * m), e = min(n, a + m);
  int gt = 0, eq = 0;
  if (keep_all) {
    gt = e - a;
  } else {
    for (int t = a; t < e; ++t) {
      const uint32_t key = keys[t];
      gt += key > thr;
      eq += key == thr;
    }
  }
  int eq_total = 0, kept_total = 0;
  const int eq_before = block_exclusive_sum(eq, wave_tot, &eq_total);
  const int take_eq = min(eq, max(0, need - eq_before));
  int rank = block_exclusive_sum(gt + take_eq, wave_tot, &kept_total);
  int32_t* kept_out = p.kept ? p.kept + unit * p.C : nullptr;
  int eq_seen = eq_before;
  for (int t = a; t < e; ++t) {
    bool keep = true;
    if (!keep_all) {
      const uint32_t key = keys[t];
      keep = key > thr;
      if (key == thr) keep = eq_seen++ < need;
    }
    if (keep) {
      if (rank >= r0 && rank < r1) {
        rows_src[rank - r0] = t;
        if (kept_out) kept_out[rank] = t;
      }
      ++rank;
    }
  }
  __syncthreads();

  // 4. copy the item's kept rows into the pages
  const int rows = r1 - r0;
  const int lpr = p.row_u4;
  const int rpp = kThreads / lpr;               // rows per pass of the workgroup
  const int sub = tid % lpr, rsel = tid / lpr;
  const int64_t tok_stride = (int64_t)p.H * lpr;
  const int64_t src0 = ((int64_t)it.b * p.C * p.H + it.kv_head) * lpr + sub;
  const int64_t v_plane = (int64_t)p.Hp * p.P * lpr;  // V rows of a page follow its K rows
  for (int base = 0; base < rows; base += kUnroll * rpp) {
    u4 kk[kUnroll], vv[kUnroll];
    int64_t dst[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int j = base + u * rpp + rsel;
      if (j < rows) {
        const int64_t src = src0 + rows_src[j] * tok_stride;
        kk[u] = p.k_new[src];
        vv[u] = p.v_new[src];
        const int pos = it.cursor + r0 + j;
        const int64_t page = p.pt_pages[it.pt_base + pos / p.P];
        dst[u] = ((page * 2 * p.Hp + it.slot) * p.P + pos % p.P) * lpr + sub;
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int j = base + u * rpp + rsel;
      if (j < rows) {
        p.pool[dst[u]] = kk[u];
        p.pool[dst[u] + v_plane] = vv[u];
      }
    }
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
  if (!a->k_new || !a->v_new || !a->scores || !a->kv_pool || !a->pt_pages || !a->items)
    return tg::fail(TG_ERR_INVALID_ARG, "NULL device pointer");
  CompressParams p;
  p.k_new = static_cast<const u4*>(a->k_new);
  p.v_new = static_cast<const u4*>(a->v_new);
  p.scores = reinterpret_cast<const uint32_t*>(a->scores);
  p.pool = static_cast<u4*>(a->kv_pool);
  p.pt_pages = a->pt_pages;
  p.items = a->items;
  p.kept = a->kept;
  p.H = g.num_kv_heads;
  p.C = a->chunk_len;
  p.Hp = g.heads_per_group;
  p.P = g.page_size;
  p.row_u4 = g.head_dim * (a->dtype == TG_F32 ? 4 : 2) / 16;
  const size_t lds = (size_t)a->chunk_len * sizeof(uint32_t);
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  static_assert(kBins == kThreads, "one histogram bin per thread");
  if (lds > 32768) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(tg_compress_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "compress LDS attribute: %s", hipGetErrorString(e));
  }
  hipLaunchKernelGGL(tg_compress_kernel, dim3(a->num_items), dim3(kThreads), lds, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "compress launch failed: %s", hipGetErrorString(e));
  return TG_OK;
}
