// Ragged paged split-KV decode attention for gfx950 (MI355X).
//
// One decode step of one layer over Tangram's ragged cache (Section 4.2 of
// arXiv 2606.06302): every KV head h of request b keeps its own number of
// retained rows, stored in the pages of its head group.  The host partition
// (tg_build_plan, Algorithm 1's proportional rule or the sequential fill)
// cuts every (b, h) into page-aligned chunks and places them on n_bins bins;
// worker k of the launch runs bin k (a wave in the matrix-core kernel, a
// workgroup in the generic one).  A chunk of a split unit writes an fp32
// partial (o, lse), and the partials of every split unit are combined with a
// log-sum-exp merge (split-KV decoding, Section 2.2.3): by tg_merge_kernel,
// launched right after on the same stream, or, with arrival counters, inside
// the matrix-core launch by the piece that finishes last.  The in-launch merge
// orders partials and counters with device-scope stores, loads and atomics
// only: a fence for ordinary stores would write back and invalidate the whole
// L2 of an XCD.
//
// Open-ended items (the chunk that ends a unit in a plan built for several
// steps) run to the unit's live length, and can append the step's new token
// themselves: the row is taken from the token buffer instead of the pool,
// then stored into the pool, and the live length advanced, at the item's end.
//
// The generic kernel deals the pages of an item round-robin to the 4 waves of
// the workgroup; every wave keeps its own online-softmax state and the states
// are merged through LDS at the end of the item.  The wave index is made
// wave-uniform (readfirstlane) so that all item/page bookkeeping is scalar.
#include <hip/hip_runtime.h>

#include <array>
#include <cmath>
#include <cstring>
#include <mutex>
#include <utility>

#include "tg_device.h"
#include "tg_internal.h"

namespace {

using namespace tgd;

constexpr int kWaves = 4;
constexpr int kBlock = 64 * kWaves;
constexpr int kPage = 16;

// 16 bytes as a native vector so staged page data stays in VGPRs
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

template <typename T>
struct Store;
template <>
struct Store<float> {
  static constexpr int kBytes = 4;
};
template <>
struct Store<uint16_t> {
  static constexpr int kBytes = 2;
};

// Partial dot product of one 16-byte chunk of K with the matching q chunk.
template <typename T>
__device__ __forceinline__ float chunk_dot(const u4& k, const u4& q, float acc);
template <>
__device__ __forceinline__ float chunk_dot<uint16_t>(const u4& k, const u4& q, float acc) {
  acc = dot2_bf16(k.x, q.x, acc);
  acc = dot2_bf16(k.y, q.y, acc);
  acc = dot2_bf16(k.z, q.z, acc);
  acc = dot2_bf16(k.w, q.w, acc);
  return acc;
}
template <>
__device__ __forceinline__ float chunk_dot<float>(const u4& k, const u4& q, float acc) {
  acc = fmaf(__uint_as_float(k.x), __uint_as_float(q.x), acc);
  acc = fmaf(__uint_as_float(k.y), __uint_as_float(q.y), acc);
  acc = fmaf(__uint_as_float(k.z), __uint_as_float(q.z), acc);
  acc = fmaf(__uint_as_float(k.w), __uint_as_float(q.w), acc);
  return acc;
}

// Unpack a 16-byte chunk of V into fp32.
template <typename T>
__device__ __forceinline__ void chunk_unpack(const u4& v, float* f);
template <>
__device__ __forceinline__ void chunk_unpack<uint16_t>(const u4& v, float* f) {
  f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x);
  f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
  f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z);
  f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
}
template <>
__device__ __forceinline__ void chunk_unpack<float>(const u4& v, float* f) {
  f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
  f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
}

template <typename T>
__device__ __forceinline__ void store_out(T* dst, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* dst, float v) { *dst = v; }
template <>
__device__ __forceinline__ void store_out<uint16_t>(uint16_t* dst, float v) { *dst = f32_to_bf16(v); }

// four consecutive outputs, one 16- or 8-byte store (dst 16- or 8-byte aligned)
template <typename T>
__device__ __forceinline__ void store_out4(T* dst, float v0, float v1, float v2, float v3);
template <>
__device__ __forceinline__ void store_out4<float>(float* dst, float v0, float v1, float v2, float v3) {
  *reinterpret_cast<float4*>(dst) = make_float4(v0, v1, v2, v3);
}
template <>
__device__ __forceinline__ void store_out4<uint16_t>(uint16_t* dst, float v0, float v1, float v2, float v3) {
  *reinterpret_cast<uint2*>(dst) = make_uint2(uint32_t(f32_to_bf16(v0)) | (uint32_t(f32_to_bf16(v1)) << 16),
                                              uint32_t(f32_to_bf16(v2)) | (uint32_t(f32_to_bf16(v3)) << 16));
}

struct DecodeParams {
  const void* q;
  const u4* pool;            // 16-byte view of the page pool
  const int32_t* pt_pages;
  const tg_work_item* items;
  const int32_t* bin_offsets;
  const int32_t* unit_splits;
  const int32_t* unit_partial_base;
  void* out;
  float* lse;
  float* part_o;             // [num_partials][gqa][d]
  float* part_lse;           // [num_partials][gqa]
  int64_t page_chunks;       // 16-byte chunks per physical page
  int32_t heads_per_group;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t n_bins;
  int32_t gqa;               // query heads per KV head
  uint64_t* timestamps;      // [n_bins][2] start / end stamps, or NULL
  const int32_t* live;       // live lengths of this layer: live[b * live_stride + h], or NULL
  int32_t live_stride;
  float scale_log2;          // sm_scale * log2(e)
  float scale;               // sm_scale
  int32_t* merge_counters;   // [B*H] arrival counters of the in-launch merge, or NULL
  // in-launch decode-token append (open items only), or append_k == NULL
  const u4* append_k;        // [B][H] token rows, 16-byte chunks
  const u4* append_v;
  u4* pool_w;                // the pool, written at the appended rows only
  int32_t* live_w;           // = live, written by the open items
  int32_t* append_full;      // set when a unit cannot take its token, or NULL
};

// An open-ended item (tok_end = -capacity) runs to the head's live length n,
// kept within [tok_begin + 1, capacity]; without live lengths, to capacity.
// With the in-launch append, an open item with tok_begin <= n < capacity
// takes the new token as entry n and runs to n + 1 (*arow = n); otherwise
// *arow = -1, and -2 for an open item that cannot take the token.
__device__ __forceinline__ int resolve_open(int tok_begin, int tok_end, int n, bool append, int* arow) {
  const int cap = -tok_end;
  if (append && n >= tok_begin && n < cap) {
    *arow = n;
    return n + 1;
  }
  *arow = append ? -2 : -1;
  return min(max(n, tok_begin + 1), cap);
}

__device__ __forceinline__ int resolve_end(int tok_begin, int tok_end, int b, int h, const DecodeParams& p,
                                           int* arow) {
  *arow = -1;
  if (tok_end >= 0) return tok_end;
  const int n = p.live ? p.live[(int64_t)b * p.live_stride + h] : -tok_end;
  return resolve_open(tok_begin, tok_end, n, p.append_k != nullptr, arow);
}

__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// End of an item: combine the per-wave states (m, l in LDS [kWaves][G],
// accumulators at acc + w*acc_stride + g*D + e) and write the final output or
// this chunk's fp32 partial (normalised o and its lse).  Called by the whole
// workgroup after a barrier.
template <typename T, int G, int D>
__device__ __forceinline__ void finish_item(const DecodeParams& p, const tg_work_item& item, const float (*sm_m)[G],
                                            const float (*sm_l)[G], const float* acc, int acc_stride) {
  const float cs = p.scale_log2;
  const int qh0 = item.kv_head * G;
  for (int o = threadIdx.x; o < G * D; o += kBlock) {
    const int g = o / D, e = o % D;
    float M = sm_m[0][g];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) M = fmaxf(M, sm_m[w][g]);
    float L = 0.f, A = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float f = fast_exp2((sm_m[w][g] - M) * cs);   // 0 for a wave that saw no rows
      L = fmaf(sm_l[w][g], f, L);
      A = fmaf(acc[w * acc_stride + g * D + e], f, A);
    }
    const float O = A / L;
    const float lse_nat = M * p.scale + logf(L);
    if (item.out_idx < 0) {
      store_out<T>(static_cast<T*>(p.out) + ((int64_t)item.b * p.num_q_heads + qh0 + g) * D + e, O);
      if (p.lse && e == 0) p.lse[(int64_t)item.b * p.num_q_heads + qh0 + g] = lse_nat;
    } else {
      p.part_o[((int64_t)item.out_idx * G + g) * D + e] = O;
      if (e == 0) p.part_lse[(int64_t)item.out_idx * G + g] = lse_nat;
    }
  }
}

// ---------------------------------------------------------------------------
// Generic kernel: any head_dim in {64, 128}, fp32 or bf16, 1..16 query heads per
// KV head.  A page slab (P=16 rows of one head, d*sizeof(T) bytes each) is read
// with one 16-byte load per lane per 64 chunks; lane l owns chunk l % CPR of
// token row l / CPR (CPR = 16-byte chunks per row).  q.k uses v_dot2_f32_bf16
// on raw bf16 pairs (fp32 FMAs for fp32 data) and a DPP all-reduce over the CPR
// lanes of a row; the per-page max uses the gfx950 permlane16/32 swaps.
template <typename T, int D>
struct Tile {
  static constexpr int kRowBytes = D * Store<T>::kBytes;
  static constexpr int kCPR = kRowBytes / 16;
  static constexpr int kEPC = 16 / Store<T>::kBytes;
  static constexpr int kTPL = 64 / kCPR;
  static constexpr int kSlots = kPage / kTPL;
  static constexpr int kSlabChunks = kPage * kCPR;
  static_assert(kCPR == 8 || kCPR == 16 || kCPR == 32, "unsupported row size");
};

template <typename T, int D, int GQA>
__global__ void __launch_bounds__(kBlock) tg_decode_kernel(DecodeParams p, const tg_work_item* __restrict__ items,
                                                          const int32_t* __restrict__ pt_pages,
                                                          const int32_t* __restrict__ bin_offsets,
                                                          const u4* __restrict__ pool) {
  using TL = Tile<T, D>;
  constexpr int CPR = TL::kCPR, EPC = TL::kEPC, TPL = TL::kTPL, NS = TL::kSlots;

  __shared__ float sm_m[kWaves][GQA];
  __shared__ float sm_l[kWaves][GQA];
  __shared__ float sm_acc[kWaves][GQA][D];

  const int lane = threadIdx.x & 63;
  const int wave = wave_id();
  const int c = lane % CPR;
  const int r = lane / CPR;
  const int it_begin = bin_offsets[blockIdx.x], it_end = bin_offsets[blockIdx.x + 1];
  const float cs = p.scale_log2;
  const uint64_t t_start = __builtin_amdgcn_s_memrealtime();

  for (int it = it_begin; it < it_end; ++it) {
    tg_work_item item = items[it];
    int arow;   // entry that takes the appended token, or < 0
    item.tok_end = resolve_end(item.tok_begin, item.tok_end, item.b, item.kv_head, p, &arow);
    const int qh0 = item.kv_head * GQA;
    const int64_t toff = ((int64_t)item.b * p.num_kv_heads + item.kv_head) * CPR;   // token row, in chunks
    u4 qv[GQA];
    {
      const u4* qbase = reinterpret_cast<const u4*>(static_cast<const T*>(p.q) +
                                                    ((int64_t)item.b * p.num_q_heads + qh0) * D);
#pragma unroll
      for (int g = 0; g < GQA; ++g) qv[g] = qbase[g * CPR + c];
    }
    float m[GQA], l[GQA], acc[GQA][EPC];
#pragma unroll
    for (int g = 0; g < GQA; ++g) {
      m[g] = -INFINITY;
      l[g] = 0.f;
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[g][e] = 0.f;
    }
    const int ntok = item.tok_end - item.tok_begin;
    const int npages = (ntok + kPage - 1) / kPage;
    const int32_t* pt = pt_pages + item.pt_base + item.tok_begin / kPage;
    const int64_t slab_k = (int64_t)item.slot * TL::kSlabChunks;
    const int64_t slab_v = ((int64_t)p.heads_per_group + item.slot) * TL::kSlabChunks;
    for (int pi = wave; pi < npages; pi += kWaves) {
      u4 kc[NS], vc[NS];
      {
        const int64_t pg = (int64_t)pt[pi] * p.page_chunks;
        const u4* kb = pool + pg + slab_k + lane;
        const u4* vb = pool + pg + slab_v + lane;
#pragma unroll
        for (int j = 0; j < NS; ++j) {
          kc[j] = kb[j * 64];
          vc[j] = vb[j * 64];
        }
      }
      if (arow >= 0 && pi == npages - 1) {   // the appended entry is the item's last: its row comes from the token
#pragma unroll
        for (int j = 0; j < NS; ++j)
          if (j * TPL + r == (arow & (kPage - 1))) {
            kc[j] = p.append_k[toff + c];
            vc[j] = p.append_v[toff + c];
          }
      }
      const int nvalid = min(kPage, ntok - pi * kPage);
      float s[NS][GQA];
#pragma unroll
      for (int j = 0; j < NS; ++j) {
#pragma unroll
        for (int g = 0; g < GQA; ++g) {
          float d = chunk_dot<T>(kc[j], qv[g], 0.f);
          if constexpr (CPR == 32) d = swap16_sum(group_sum<16>(d));
          else d = group_sum<CPR>(d);
          s[j][g] = d;
        }
      }
      if (nvalid < kPage) {
#pragma unroll
        for (int j = 0; j < NS; ++j) {
          const bool ok = j * TPL + r < nvalid;
#pragma unroll
          for (int g = 0; g < GQA; ++g) s[j][g] = ok ? s[j][g] : -INFINITY;
          if (!ok) vc[j] = u4(0u);
        }
      }
#pragma unroll
      for (int g = 0; g < GQA; ++g) {
        float mx = s[0][g];
#pragma unroll
        for (int j = 1; j < NS; ++j) mx = fmaxf(mx, s[j][g]);
        mx = rows_max<CPR>(mx);
        if (mx > m[g]) {
          const float alpha = fast_exp2((m[g] - mx) * cs);
          m[g] = mx;
          l[g] *= alpha;
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[g][e] *= alpha;
        }
      }
#pragma unroll
      for (int j = 0; j < NS; ++j) {
        float vf[EPC];
        chunk_unpack<T>(vc[j], vf);
#pragma unroll
        for (int g = 0; g < GQA; ++g) {
          const float pj = fast_exp2(fmaf(s[j][g], cs, -m[g] * cs));
          l[g] += pj;
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[g][e] = fmaf(pj, vf[e], acc[g][e]);
        }
      }
    }
#pragma unroll
    for (int g = 0; g < GQA; ++g) {
      l[g] = rows_sum<CPR>(l[g]);
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[g][e] = rows_sum<CPR>(acc[g][e]);
    }
    if (lane == 0) {
#pragma unroll
      for (int g = 0; g < GQA; ++g) {
        sm_m[wave][g] = m[g];
        sm_l[wave][g] = l[g];
      }
    }
    if (r == 0) {
#pragma unroll
      for (int g = 0; g < GQA; ++g)
#pragma unroll
        for (int e = 0; e < EPC; ++e) sm_acc[wave][g][c * EPC + e] = acc[g][e];
    }
    __syncthreads();
    finish_item<T, GQA, D>(p, item, sm_m, sm_l, &sm_acc[0][0][0], GQA * D);
    if (arow >= 0) {   // the token becomes entry arow of the cache; every thread read the length above
      if (threadIdx.x < 2 * CPR) {
        const bool is_k = threadIdx.x < CPR;
        const int ch = threadIdx.x % CPR;
        const int64_t pg = (int64_t)pt_pages[item.pt_base + arow / kPage] * p.page_chunks;
        p.pool_w[pg + (is_k ? slab_k : slab_v) + (arow % kPage) * CPR + ch] =
            is_k ? p.append_k[toff + ch] : p.append_v[toff + ch];
      }
      if (threadIdx.x == 0) p.live_w[(int64_t)item.b * p.live_stride + item.kv_head] = arow + 1;
    } else if (arow == -2 && threadIdx.x == 0 && p.append_full) {
      *p.append_full = 1;
    }
    __syncthreads();
  }
  if (p.timestamps && threadIdx.x == 0) {   // one lane, vector stores
    p.timestamps[2 * blockIdx.x] = t_start;
    p.timestamps[2 * blockIdx.x + 1] = __builtin_amdgcn_s_memrealtime();
  }
}

// ---------------------------------------------------------------------------
// Fast path for bf16 and head_dim 128, any gqa G in 1..16: matrix cores.
//
// Every wave is an independent worker: bin 4*blockIdx.x + wave of the plan.
// There is no barrier and no cross-wave merge; a wave runs its bin's items one
// after the other, page by page.
//
// Data movement.  Pages stream from HBM straight into a ring of R page buffers
// in the wave's own LDS with gfx950's global_load_lds_dwordx4 (no staging
// registers): page k+R-1 is issued before page k is computed, so R-1 pages
// (8 KiB each) stay in flight while the wave computes.  The DMA is issued from
// inline assembly, invisible to the compiler's wait-count pass (which would
// otherwise drain every load before each LDS read), and the wave waits for
// page k with an explicit vmcnt that counts the DMA instructions issued after
// it; any other vector memory operation issued later (output stores) only
// makes that wait stricter.  Page ids and work items are read through the
// constant address space, i.e. with scalar loads, which the vector memory
// counter does not see.  The queries of an item are DMA'd with its first page
// into one of R-1 per-wave q slots and moved to registers when the item starts.
//
// Arithmetic, per 16-token page, with the query heads of the KV head as the
// 16 columns of the MFMA tiles (columns past G repeat a real head and are
// never stored):
//   * S^T[16 tok][16 heads] = K q^T: 4 x v_mfma_f32_16x16x32_bf16, A = K rows
//     read from LDS (16 bytes per lane), B = q from registers.  Lane
//     (col, rb) = (lane % 16, lane / 16) receives tokens 4rb..4rb+3 of head col.
//   * online softmax on those 4 values per lane; the row max and sum of a head
//     combine the 4 lanes of its column with the gfx950 permlane swaps.  The
//     running max is only raised when a page exceeds it by more than 8 (in
//     log2 units), so rescales are rare and p stays <= 2^8.
//   * O^T[16 dims][16 heads] += V^T P^T: 8 x v_mfma_f32_16x16x16_bf16, one per
//     16 dims.  P^T is the S^T tile of the same lane rounded to bf16 (the
//     result layout of the first product is the operand layout of the second),
//     and V^T comes from LDS with ds_read_b64_tr_b16, whose 4x4 lane transpose
//     turns row-major V rows into the 4-consecutive-token operand.
//   * LDS layout: chunk c (16 bytes) of token row r sits at position c ^ r in
//     the K slab and at c ^ (2r mod 16) in the V slab (the DMA lanes pick their
//     source chunk accordingly), so both operand reads are bank-conflict free.
// The accumulator of a lane belongs to one head, so rescaling and the final
// normalisation need no cross-lane traffic.
constexpr int kFastWorkers = kWaves;   // bins per workgroup in the fast path

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4_vs __attribute__((__vector_size__(4 * sizeof(__bf16))));

#define TG_CONST __attribute__((address_space(4)))
#define TG_LDS __attribute__((address_space(3)))

__device__ __forceinline__ uint32_t lds_address(const void* ptr) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const TG_LDS void*)ptr));
}

// 16 bytes per lane from global memory into LDS at m0_base + 16 * lane.  A
// decode step reads every retained K/V byte exactly once, so the loads carry
// the non-temporal (streaming) policy, at device scope.
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t m0_base) {
  asm volatile("global_load_lds_dwordx4 %0, off nt sc1" ::"v"(src), "{m0}"(m0_base) : "memory");
}

// vmcnt(n) with expcnt/lgkmcnt left alone; the memory clobber keeps LDS reads
// below it.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ void wait_lgkmcnt0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// field-wise copy: the implicit copy constructor cannot bind a constant-space object
// (live lengths too: the open item that appends writes its length only after
// its last scalar read of it)
__device__ __forceinline__ tg_work_item load_item(const TG_CONST tg_work_item* src, const DecodeParams& p, int* arow) {
  tg_work_item r;
  r.pt_base = src->pt_base;
  r.b = src->b;
  r.kv_head = src->kv_head;
  r.slot = src->slot;
  r.tok_begin = src->tok_begin;
  r.tok_end = src->tok_end;
  r.out_idx = src->out_idx;
  *arow = -1;
  if (r.tok_end < 0) {
    const TG_CONST int32_t* live = (const TG_CONST int32_t*)p.live;
    const int n = live ? live[(int64_t)r.b * p.live_stride + r.kv_head] : -r.tok_end;
    r.tok_end = resolve_open(r.tok_begin, r.tok_end, n, p.append_k != nullptr, arow);
  }
  return r;
}

// two fp32 values as one 64-bit word (lo first, as they sit in memory)
__device__ __forceinline__ uint64_t pack_f32x2(float lo, float hi) {
  return (uint64_t)__float_as_uint(lo) | ((uint64_t)__float_as_uint(hi) << 32);
}

__device__ __forceinline__ f32x4 mfma_qk(const u4& a, const u4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0,
                                                 0);
}
__device__ __forceinline__ f32x4 mfma_pv(const s16x4& a, const s16x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
// Lane l of each 16-lane block receives element l % 4 of the 8-byte rows
// addressed by lanes l/4, l/4 + 4, l/4 + 8, l/4 + 12 of the block.
__device__ __forceinline__ s16x4 lds_read_tr16(const void* ptr) {
  return __builtin_bit_cast(s16x4, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((TG_LDS bf16x4_vs*)ptr));
}

// This file is built with -mllvm -amdgpu-mfma-vgpr-form: the accumulators stay
// in VGPRs, where the rescale multiplies them in place, instead of being
// copied between AGPRs and VGPRs on every page.
template <int QMAX>   // 8 or 16: the q slots hold up to QMAX query heads
__global__ void __launch_bounds__(kBlock) tg_decode_mfma_kernel(DecodeParams p, const tg_work_item* __restrict__ items_g,
                                                               const int32_t* __restrict__ pt_g,
                                                               const int32_t* __restrict__ bin_offsets_g,
                                                               const u4* __restrict__ pool) {
  constexpr int D = 128;
  constexpr int R = QMAX <= 8 ? 4 : 3;   // LDS page buffers per wave
  constexpr int NQ = R - 1;              // LDS query buffers per wave
  constexpr int kQChunks = QMAX * (D / 8);
  constexpr int kDma = 8;                // DMA instructions per page: 4 K + 4 V
  constexpr float kSlack = 8.0f;
  static_assert(kPage == 16, "one page is one 4 KiB K slab and one 4 KiB V slab");

  __shared__ u4 sm_ring[kWaves][R][512];   // page: K slab, then V slab
  __shared__ u4 sm_q[kWaves][NQ][kQChunks];

  const TG_CONST tg_work_item* const items = (const TG_CONST tg_work_item*)items_g;
  const TG_CONST int32_t* const pt = (const TG_CONST int32_t*)pt_g;
  const TG_CONST int32_t* const bin_offsets = (const TG_CONST int32_t*)bin_offsets_g;

  const int lane = threadIdx.x & 63;
  const int wave = wave_id();
  const int bin = blockIdx.x * kFastWorkers + wave;
  if (bin >= p.n_bins) return;
  const uint64_t t_start = __builtin_amdgcn_s_memrealtime();
  const int it_begin = bin_offsets[bin], it_end = bin_offsets[bin + 1];
  if (it_begin >= it_end) {
    if (p.timestamps && lane == 0) {   // one lane, vector stores
      p.timestamps[2 * bin] = t_start;
      p.timestamps[2 * bin + 1] = t_start;
    }
    return;
  }
  const int G = p.gqa;
  const int col = lane & 15;            // head column of the MFMA tiles
  const int rb = lane >> 4;             // row block: tokens / dims 4rb..4rb+3
  const int hq = col < G ? col : col % G;
  const float cs = p.scale_log2;
  const uint32_t ring_lds = lds_address(&sm_ring[wave][0][0]);
  const uint32_t q_lds = lds_address(&sm_q[wave][0][0]);
  const u4* const qsrc = static_cast<const u4*>(p.q);
  const int nq = G * (D / 8);           // 16-byte chunks of one item's queries

  // DMA cursor over every page of every item of the bin; it caches the
  // item's page count, table base, slot and query offset.
  struct Cursor {
    int it, pi, np, slot, arow;
    int64_t pbase, qoff;
  };
  auto enter = [&](Cursor& cu, int it) {
    int arow;
    const tg_work_item im = load_item(items + it, p, &arow);
    cu.it = it;
    cu.pi = 0;
    cu.np = (im.tok_end - im.tok_begin + kPage - 1) / kPage;
    cu.slot = im.slot;
    cu.arow = arow >= 0 ? arow & (kPage - 1) : -1;   // row of the last page that takes the new token
    cu.pbase = im.pt_base + im.tok_begin / kPage;
    cu.qoff = ((int64_t)im.b * p.num_q_heads + (int64_t)im.kv_head * G) * (D / 8);
  };
  auto advance = [&](Cursor& cu) {   // false (cursor unchanged) past the bin's last page
    if (cu.pi + 1 < cu.np) {
      ++cu.pi;
      return true;
    }
    if (cu.it + 1 < it_end) {
      enter(cu, cu.it + 1);
      return true;
    }
    return false;
  };
  // queries (on an item's first page), then the page's K slab, then its V slab
  auto issue = [&](const Cursor& cu, int32_t id, int ring) {
    if (cu.pi == 0) {
      const u4* qb = qsrc + cu.qoff;
      const uint32_t dst = q_lds + ((cu.it - it_begin) % NQ) * (kQChunks * 16);
#pragma unroll
      for (int j = 0; j < kQChunks / 64; ++j)
        if (j * 64 < nq) lds_dma16(qb + min(j * 64 + lane, nq - 1), dst + j * 1024);
    }
    const u4* base = pool + (int64_t)id * p.page_chunks;
    const u4* kb = base + cu.slot * 256;
    const u4* vb = base + (p.heads_per_group + cu.slot) * 256;
    const uint32_t dst = ring_lds + ring * 8192;
    if (cu.arow >= 0 && cu.pi == cu.np - 1) {   // the page that takes the new token: that row from the token
      const int64_t toff = ((int64_t)items[cu.it].b * p.num_kv_heads + items[cu.it].kv_head) * (D / 8);
      const u4* tk = p.append_k + toff;
      const u4* tv = p.append_v + toff;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = j * 4 + (lane >> 4);
        const int pos = lane & 15;
        lds_dma16(r == cu.arow ? tk + (pos ^ r) : kb + r * 16 + (pos ^ r), dst + j * 1024);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = j * 4 + (lane >> 4);
        const int pos = lane & 15;
        const int c = pos ^ ((2 * r) & 15);
        lds_dma16(r == cu.arow ? tv + c : vb + r * 16 + c, dst + 4096 + j * 1024);
      }
      return;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = j * 4 + (lane >> 4);   // token row written by this lane
      const int pos = lane & 15;           // chunk position within the row
      lds_dma16(kb + r * 16 + (pos ^ r), dst + j * 1024);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = j * 4 + (lane >> 4);
      const int pos = lane & 15;
      lds_dma16(vb + r * 16 + (pos ^ ((2 * r) & 15)), dst + 4096 + j * 1024);
    }
  };

  Cursor d;
  enter(d, it_begin);
  bool d_live = true;
  int32_t d_id = pt[d.pbase];
#pragma unroll
  for (int r = 0; r < R - 1; ++r) {
    if (d_live) {
      issue(d, d_id, r);
      d_live = advance(d);
      if (d_live) d_id = pt[d.pbase + d.pi];
    }
  }

  // lane-constant parts of the operand addresses
  const int k_off = col * 16;                                  // A of q.k: token row col
  const int v_tok = lane >> 2;                                 // source row of the transposed read
  const int v_off = 4096 + v_tok * 256 + (lane & 3) * 8;       // bytes within the page buffer
  const int v_swz = v_tok & 7;

  int it = it_begin, pi = 0, np = 0, ntok = 0, k = 0, arow = -1;
  tg_work_item item;
  u4 qv[4];
  float m = -INFINITY, l = 0.f;
  f32x4 acc[8];
  for (;;) {
    if (pi == 0) {   // item start: its queries were DMA'd just before its first page
      item = load_item(items + it, p, &arow);
      ntok = item.tok_end - item.tok_begin;
      np = (ntok + kPage - 1) / kPage;
      if (d_live)
        wait_vmcnt<kDma * (R - 1)>();
      else
        wait_vmcnt<0>();
      const u4* qrow = &sm_q[wave][(it - it_begin) % NQ][hq * 16 + rb];
#pragma unroll
      for (int c = 0; c < 4; ++c) qv[c] = qrow[4 * c];
      wait_lgkmcnt0();   // the slot may be refilled by the DMA issued next
      m = -INFINITY;
      l = 0.f;
#pragma unroll
      for (int mm = 0; mm < 8; ++mm) acc[mm] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    if (d_live) {   // keep R-1 pages in flight: issue page k+R-1, then wait for page k
      issue(d, d_id, (k + R - 1) % R);
      d_live = advance(d);
      if (d_live) d_id = pt[d.pbase + d.pi];
      wait_vmcnt<kDma * (R - 1)>();
    } else {
      wait_vmcnt<0>();
    }
    const int rs = k % R;
    const u4* const kbuf = &sm_ring[wave][rs][0];
    const char* const pbuf = reinterpret_cast<const char*>(&sm_ring[wave][rs][0]);
    const int nvalid = min(kPage, ntok - pi * kPage);

    // S^T = K q^T
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 4; ++c) s = mfma_qk(kbuf[k_off + ((4 * c + rb) ^ col)], qv[c], s);
    float sv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) sv[i] = 4 * rb + i < nvalid ? s[i] : -INFINITY;
    float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    mx = swap32_max(swap16_max(mx));
    const bool raise = (mx - m) * cs > kSlack;
    if (__any(raise)) {
      const float m_new = raise ? mx : m;
      const float alpha = fast_exp2((m - m_new) * cs);   // 0 when m was -inf
      l *= alpha;
      m = m_new;
#pragma unroll
      for (int mm = 0; mm < 8; ++mm) acc[mm] *= alpha;
    }
    const float mcs = m * cs;
    s16x4 pb;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float pk = fast_exp2(fmaf(sv[i], cs, -mcs));
      l += pk;
      pb[i] = (short)f32_to_bf16(pk);
    }
    // O^T += V^T P^T
    const bool partial = nvalid < kPage;
#pragma unroll
    for (int mm = 0; mm < 8; ++mm) {
      s16x4 a = lds_read_tr16(pbuf + v_off + ((mm ^ v_swz) << 5));
      if (partial) {   // rows past the retained length may hold anything
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (4 * rb + j >= nvalid) a[j] = 0;
      }
      acc[mm] = mfma_pv(a, pb, acc[mm]);
    }
    ++k;
    if (++pi < np) continue;

    if (arow >= 0) {
      // the new token becomes entry arow of the cache: its rows are in this
      // page's LDS buffer (refilled only by the next issue), 16 lanes for K
      // and 16 for V, stored with ordinary vector stores, which the DMA waits
      // above only count as extra (later) operations
      const int r = arow & (kPage - 1);
      const int64_t pg = (int64_t)pt[item.pt_base + arow / kPage] * p.page_chunks;
      if (lane < 32) {
        const int ch = lane & 15;
        const bool is_k = lane < 16;
        const u4 row = is_k ? kbuf[r * 16 + (ch ^ r)] : kbuf[256 + r * 16 + (ch ^ ((2 * r) & 15))];
        p.pool_w[pg + (is_k ? item.slot : p.heads_per_group + item.slot) * 256 + r * 16 + ch] = row;
      }
      if (lane == 0) p.live_w[(int64_t)item.b * p.live_stride + item.kv_head] = arow + 1;
    } else if (arow == -2 && lane == 0 && p.append_full) {
      *p.append_full = 1;
    }

    // item end: the head's sum over all 16 token rows, then normalise and store
    l = swap32_sum(swap16_sum(l));
    if (col < G) {
      const float lse_nat = m * p.scale + logf(l);
      const float inv = 1.f / l;
      const int qh = item.kv_head * G + col;
      if (item.out_idx < 0) {
        uint2* orow = reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.out) +
                                               ((int64_t)item.b * p.num_q_heads + qh) * D + 4 * rb);
#pragma unroll
        for (int mm = 0; mm < 8; ++mm) {
          const f32x4 o = acc[mm] * inv;
          orow[mm * 4] = make_uint2(uint32_t(f32_to_bf16(o[0])) | (uint32_t(f32_to_bf16(o[1])) << 16),
                                    uint32_t(f32_to_bf16(o[2])) | (uint32_t(f32_to_bf16(o[3])) << 16));
        }
        if (p.lse && rb == 0) p.lse[(int64_t)item.b * p.num_q_heads + qh] = lse_nat;
      } else if (p.merge_counters) {
        // read in this launch by whichever worker merges the unit, maybe on
        // another XCD: device-scope stores, written through to where every
        // XCD's device-scope loads read
        uint64_t* prow = reinterpret_cast<uint64_t*>(p.part_o + ((int64_t)item.out_idx * G + col) * D + 4 * rb);
#pragma unroll
        for (int mm = 0; mm < 8; ++mm) {
          const f32x4 o = acc[mm] * inv;
          __hip_atomic_store(prow + mm * 8, pack_f32x2(o[0], o[1]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(prow + mm * 8 + 1, pack_f32x2(o[2], o[3]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (rb == 0)
          __hip_atomic_store(p.part_lse + (int64_t)item.out_idx * G + col, lse_nat, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
      } else {
        f32x4* prow = reinterpret_cast<f32x4*>(p.part_o + ((int64_t)item.out_idx * G + col) * D + 4 * rb);
#pragma unroll
        for (int mm = 0; mm < 8; ++mm) prow[mm * 4] = acc[mm] * inv;
        if (rb == 0) p.part_lse[(int64_t)item.out_idx * G + col] = lse_nat;
      }
    }
    pi = 0;
    if (++it == it_end) break;
  }
  wait_vmcnt<0>();   // every page and every partial of this worker is complete

  // In-launch log-sum-exp merge (split-KV decoding, Section 2.2.3).  Each split
  // piece this worker ran counts itself on its unit's arrival counter; the
  // piece that arrives last merges the unit's partials and resets the counter
  // for the next call.  The partials were written with device-scope stores and
  // are complete (the wait above) before the worker's increments; the merging
  // worker reads them with device-scope loads issued after its increment
  // returned.  This is the ordering a release/acquire pair gives for data
  // written and read by device-scope atomics, without the writeback and
  // invalidation of a whole L2 that a fence for ordinary data needs.
  if (p.merge_counters) {
    const TG_CONST int32_t* const unit_splits = (const TG_CONST int32_t*)p.unit_splits;
    const TG_CONST int32_t* const unit_base = (const TG_CONST int32_t*)p.unit_partial_base;
    // the split items of the bin, up to kBatch at a time: all their arrivals
    // go out before the first result is waited for, so a worker pays one
    // round trip for them, not one per item
    constexpr int kBatch = 4;
    int it2 = it_begin;
    while (it2 < it_end) {
      int su[kBatch], nb = 0;   // item indices of this batch's split items
      for (; it2 < it_end && nb < kBatch; ++it2)
        if (items[it2].out_idx >= 0) su[nb++] = it2;
      if (nb == 0) break;
      int arrived[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        arrived[j] = 0;
        if (j < nb && lane == 0) {
          const int u = items[su[j]].b * p.num_kv_heads + items[su[j]].kv_head;
          arrived[j] = __hip_atomic_fetch_add(p.merge_counters + u, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        if (j >= nb) break;
        const int b = items[su[j]].b, h = items[su[j]].kv_head;
        const int u = b * p.num_kv_heads + h;
        const int s = unit_splits[u], base = unit_base[u];
        if (__builtin_amdgcn_readfirstlane(arrived[j]) != s - 1) continue;
        if (col < G) {
          float mr = -INFINITY, L = 0.f;
          f32x4 A[8];
#pragma unroll
          for (int mm = 0; mm < 8; ++mm) A[mm] = f32x4{0.f, 0.f, 0.f, 0.f};
          // up to kSplitBatch partials are requested before the first is
          // used: one round trip for a unit of that many splits (indices past
          // the last re-read it, and selects discard their steps)
          constexpr int kSplitBatch = 4;
          for (int i0 = 0; i0 < s; i0 += kSplitBatch) {
            float lv[kSplitBatch];
            f32x4 ov[kSplitBatch][8];
#pragma unroll
            for (int jj = 0; jj < kSplitBatch; ++jj) {
              const int64_t pidx = (int64_t)base + min(i0 + jj, s - 1);
              lv[jj] = __hip_atomic_load(p.part_lse + pidx * G + col, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              const uint64_t* prow = reinterpret_cast<const uint64_t*>(p.part_o + (pidx * G + col) * D + 4 * rb);
#pragma unroll
              for (int mm = 0; mm < 8; ++mm) {
                const uint64_t lo = __hip_atomic_load(prow + mm * 8, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                const uint64_t hi = __hip_atomic_load(prow + mm * 8 + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                ov[jj][mm] = f32x4{__uint_as_float((uint32_t)lo), __uint_as_float((uint32_t)(lo >> 32)),
                                   __uint_as_float((uint32_t)hi), __uint_as_float((uint32_t)(hi >> 32))};
              }
            }
            // the same running-max recurrence, in the same order, as tg_merge_kernel
#pragma unroll
            for (int jj = 0; jj < kSplitBatch; ++jj) {
              const bool use = i0 + jj < s;
              const float mn = fmaxf(mr, lv[jj]);
              const float a = __expf(mr - mn), w = __expf(lv[jj] - mn);
              const float Ln = fmaf(L, a, w);
#pragma unroll
              for (int mm = 0; mm < 8; ++mm)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                  const float An = fmaf(A[mm][q], a, w * ov[jj][mm][q]);
                  A[mm][q] = use ? An : A[mm][q];
                }
              L = use ? Ln : L;
              mr = use ? mn : mr;
            }
          }
          const int qh = h * G + col;
          uint2* orow =
              reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.out) + ((int64_t)b * p.num_q_heads + qh) * D + 4 * rb);
#pragma unroll
          for (int mm = 0; mm < 8; ++mm)
            orow[mm * 4] =
                make_uint2(uint32_t(f32_to_bf16(A[mm][0] / L)) | (uint32_t(f32_to_bf16(A[mm][1] / L)) << 16),
                           uint32_t(f32_to_bf16(A[mm][2] / L)) | (uint32_t(f32_to_bf16(A[mm][3] / L)) << 16));
          if (p.lse && rb == 0) p.lse[(int64_t)b * p.num_q_heads + qh] = mr + logf(L);
        }
        if (lane == 0) __hip_atomic_store(p.merge_counters + u, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  if (p.timestamps && lane == 0) {   // one lane, vector stores
    p.timestamps[2 * bin] = t_start;
    p.timestamps[2 * bin + 1] = __builtin_amdgcn_s_memrealtime();
  }
}

// ---------------------------------------------------------------------------
// Log-sum-exp merge of the split partials of every unit (b, h) with more than
// one split: lse* = log sum_i e^{lse_i}, O = sum_i e^{lse_i - lse*} o_i.
// Grid (units, ceil(gqa*D / 1024)): each thread owns four consecutive output
// elements (16-byte partial loads) and makes a single pass with a running
// max, so the loads of consecutive splits are independent and issue back to
// back.
template <typename T, int D>
__global__ void __launch_bounds__(kBlock) tg_merge_kernel(const int32_t* __restrict__ unit_splits,
                                                         const int32_t* __restrict__ unit_base,
                                                         const float* __restrict__ part_o,
                                                         const float* __restrict__ part_lse, void* out, float* lse,
                                                         int32_t num_kv_heads, int32_t gqa) {
  const int u = blockIdx.x;
  const int s = unit_splits[u];
  const int base = unit_base[u];
  // both reads in flight together, before the exit test (the compiler would
  // otherwise sink the second behind it: two round trips instead of one)
  asm volatile("" ::"s"(s), "s"(base));
  const int o = (blockIdx.y * kBlock + threadIdx.x) * 4;
  if (s <= 1 || o >= gqa * D) return;
  const int b = u / num_kv_heads, h = u % num_kv_heads;
  const int64_t row0 = (int64_t)b * num_kv_heads * gqa + (int64_t)h * gqa;
  const int g = o / D, e = o % D;   // D is a multiple of 4: the four outputs share g
  const float* pl = part_lse + (int64_t)base * gqa + g;
  const f32x4* po = reinterpret_cast<const f32x4*>(part_o + ((int64_t)base * gqa + g) * D + e);
  float m = -INFINITY, L = 0.f;
  f32x4 A = {0.f, 0.f, 0.f, 0.f};
  // kBatch splits' loads go out before the first is used, so a unit of up to
  // kBatch splits pays one memory round trip, not one per split.  Indices past
  // the last split re-read it; their steps are computed and then discarded by
  // selects (a branch would let the compiler sink the loads behind it).
  constexpr int kBatch = 4;
  for (int i0 = 0; i0 < s; i0 += kBatch) {
    float lv[kBatch];
    f32x4 ov[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int64_t i = min(i0 + j, s - 1);
      lv[j] = pl[i * gqa];
      ov[j] = po[i * gqa * (D / 4)];
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const bool use = i0 + j < s;
      const float mn = fmaxf(m, lv[j]);
      const float a = __expf(m - mn), w = __expf(lv[j] - mn);
      const float Ln = fmaf(L, a, w);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float An = fmaf(A[q], a, w * ov[j][q]);
        A[q] = use ? An : A[q];
      }
      L = use ? Ln : L;
      m = use ? mn : m;
    }
  }
  store_out4<T>(static_cast<T*>(out) + (row0 + g) * D + e, A[0] / L, A[1] / L, A[2] / L, A[3] / L);
  if (lse && e == 0) lse[row0 + g] = m + logf(L);
}

using MergeFn = void (*)(const int32_t*, const int32_t*, const float*, const float*, void*, float*, int32_t,
                         int32_t);

MergeFn pick_merge(int dtype, int d) {
  if (dtype == TG_F32 && d == 64) return &tg_merge_kernel<float, 64>;
  if (dtype == TG_F32 && d == 128) return &tg_merge_kernel<float, 128>;
  if (dtype == TG_BF16 && d == 64) return &tg_merge_kernel<uint16_t, 64>;
  if (dtype == TG_BF16 && d == 128) return &tg_merge_kernel<uint16_t, 128>;
  return nullptr;
}

using DecodeFn = void (*)(DecodeParams, const tg_work_item*, const int32_t*, const int32_t*, const u4*);

template <typename T, int D, int... G>
constexpr auto make_decode_table(std::integer_sequence<int, G...>) {
  return std::array<DecodeFn, sizeof...(G)>{&tg_decode_kernel<T, D, G + 1>...};
}

constexpr int kMaxGqa = 16;
const std::array<DecodeFn, kMaxGqa> kDecodeF32D64 = make_decode_table<float, 64>(std::make_integer_sequence<int, kMaxGqa>{});
const std::array<DecodeFn, kMaxGqa> kDecodeF32D128 = make_decode_table<float, 128>(std::make_integer_sequence<int, kMaxGqa>{});
const std::array<DecodeFn, kMaxGqa> kDecodeBF16D64 = make_decode_table<uint16_t, 64>(std::make_integer_sequence<int, kMaxGqa>{});

DecodeFn pick_decode(int dtype, int d, int gqa) {
  if (gqa < 1 || gqa > kMaxGqa) return nullptr;
  if (dtype == TG_BF16 && d == 128) return gqa <= 8 ? &tg_decode_mfma_kernel<8> : &tg_decode_mfma_kernel<16>;
  if (dtype == TG_F32 && d == 64) return kDecodeF32D64[gqa - 1];
  if (dtype == TG_F32 && d == 128) return kDecodeF32D128[gqa - 1];
  if (dtype == TG_BF16 && d == 64) return kDecodeBF16D64[gqa - 1];
  return nullptr;
}

// bins run by one workgroup of the kernel pick_decode() selects
int workers_per_wg(int dtype, int d, int gqa) {
  (void)gqa;
  return (dtype == TG_BF16 && d == 128) ? kFastWorkers : 1;
}

int32_t check_decode_shape(const tg_geometry* g, int dtype) {
  if (int32_t rc = tg::check_geometry(g)) return rc;
  if (dtype != TG_F32 && dtype != TG_BF16) return tg::fail(TG_ERR_INVALID_ARG, "unknown dtype %d", dtype);
  if (g->page_size != kPage) return tg::fail(TG_ERR_UNSUPPORTED, "decode supports page_size 16 only (got %d)", g->page_size);
  if (g->head_dim != 64 && g->head_dim != 128)
    return tg::fail(TG_ERR_UNSUPPORTED, "decode supports head_dim 64 or 128 (got %d)", g->head_dim);
  const int gqa = g->num_q_heads / g->num_kv_heads;
  if (gqa < 1 || gqa > kMaxGqa) return tg::fail(TG_ERR_UNSUPPORTED, "decode supports 1..16 query heads per KV head");
  return TG_OK;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

// ---------------------------------------------------------------------------
// Static scratch of tg_decode_noalloc: the split partials of one call, for
// callers that cannot allocate device memory.  Every device the library runs
// on holds its own copy of this array until the process ends.  In host code
// `scratch` is only a stand-in symbol: its device address is looked up once
// per device (hipGetSymbolAddress, with that device current) and that address
// is what the kernels get.
static __device__ __align__(256) unsigned char scratch[TG_DECODE_NOALLOC_MAX_BYTES];

namespace {

constexpr int kMaxDevices = 64;
constexpr size_t kScratchCounters = 64 << 10;   // merge arrival counters: up to 16384 (request, KV head) units
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int32_t scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return tg::fail(TG_ERR_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return tg::fail(TG_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return tg::fail(TG_ERR_HIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return TG_OK;
}

// tg_decode with the partials' memory passed in: ws (ws_bytes bytes) stands for
// the caller's workspace.
int32_t decode_impl(const tg_decode_args* a, void* ws_ptr, size_t ws_bytes, void* hip_stream) {
  if (!a) return tg::fail(TG_ERR_INVALID_ARG, "args is NULL");
  if (int32_t rc = check_decode_shape(&a->geom, a->dtype)) return rc;
  const tg_geometry& g = a->geom;
  if (a->batch < 1 || a->n_bins < 1 || a->num_items < 0 || a->num_partials < 0)
    return tg::fail(TG_ERR_INVALID_ARG, "batch, n_bins must be >= 1; counts >= 0");
  if (!a->q || !a->kv_pool || !a->pt_pages || !a->items || !a->bin_offsets || !a->out)
    return tg::fail(TG_ERR_INVALID_ARG, "NULL device pointer");
  if (a->num_partials > 0 && (!a->unit_splits || !a->unit_partial_base))
    return tg::fail(TG_ERR_INVALID_ARG, "split plan needs unit_splits and unit_partial_base");
  const size_t need = tg_decode_workspace_bytes(&g, a->batch, a->num_partials);
  if (a->num_partials > 0 && (!ws_ptr || ws_bytes < need))
    return tg::fail(TG_ERR_BUFFER_TOO_SMALL, "workspace holds %zu bytes, need %zu", ws_bytes, need);
  if (!tg::aligned16({a->q, a->kv_pool, a->out, a->append_k, a->append_v, a->num_partials > 0 ? ws_ptr : nullptr}))
    return tg::fail(TG_ERR_INVALID_ARG, "device buffers must be 16-byte aligned");
  const int gqa = g.num_q_heads / g.num_kv_heads;
  const int esz = a->dtype == TG_F32 ? 4 : 2;
  const size_t o_bytes = align256((size_t)a->num_partials * gqa * g.head_dim * 4);
  char* ws = static_cast<char*>(ws_ptr);
  DecodeParams p;
  p.q = a->q;
  p.pool = static_cast<const u4*>(a->kv_pool);
  p.pt_pages = a->pt_pages;
  p.items = a->items;
  p.bin_offsets = a->bin_offsets;
  p.unit_splits = a->unit_splits;
  p.unit_partial_base = a->unit_partial_base;
  p.out = a->out;
  p.lse = a->lse;
  p.part_o = ws ? reinterpret_cast<float*>(ws) : nullptr;
  p.part_lse = ws ? reinterpret_cast<float*>(ws + o_bytes) : nullptr;
  p.page_chunks = (int64_t)g.heads_per_group * 2 * kPage * g.head_dim * esz / 16;
  p.heads_per_group = g.heads_per_group;
  p.num_q_heads = g.num_q_heads;
  p.num_kv_heads = g.num_kv_heads;
  p.n_bins = a->n_bins;
  p.gqa = gqa;
  p.timestamps = a->timestamps;
  if (a->live_len && (a->layer < 0 || a->layer >= g.num_layers))
    return tg::fail(TG_ERR_INVALID_ARG, "layer %d out of range", a->layer);
  p.live = a->live_len ? a->live_len + (int64_t)a->layer * g.num_kv_heads : nullptr;
  p.live_stride = g.num_layers * g.num_kv_heads;
  if ((a->append_k == nullptr) != (a->append_v == nullptr))
    return tg::fail(TG_ERR_INVALID_ARG, "append_k and append_v go together");
  if (a->append_k && !a->live_len) return tg::fail(TG_ERR_INVALID_ARG, "the in-launch append needs live_len");
  p.append_k = static_cast<const u4*>(a->append_k);
  p.append_v = static_cast<const u4*>(a->append_v);
  p.pool_w = static_cast<u4*>(a->kv_pool);
  p.live_w = a->append_k ? a->live_len + (int64_t)a->layer * g.num_kv_heads : nullptr;
  p.append_full = a->append_full;
  // the bf16 head_dim-128 kernel merges split units inside its launch when the
  // caller passes arrival counters; every other case merges in a second launch
  const bool fused_merge = a->merge_counters && a->num_partials > 0 && a->dtype == TG_BF16 && g.head_dim == 128;
  p.merge_counters = fused_merge ? a->merge_counters : nullptr;
  p.scale = a->sm_scale != 0.f ? a->sm_scale : 1.0f / std::sqrt((float)g.head_dim);
  p.scale_log2 = p.scale * kLog2e;
  if (a->num_items == 0) return TG_OK;
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  DecodeFn fn = pick_decode(a->dtype, g.head_dim, gqa);
  const int wpw = workers_per_wg(a->dtype, g.head_dim, gqa);
  hipLaunchKernelGGL(fn, dim3((a->n_bins + wpw - 1) / wpw), dim3(kBlock), 0, st, p, a->items, a->pt_pages,
                     a->bin_offsets, p.pool);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "decode launch failed: %s", hipGetErrorString(e));
  if (a->num_partials > 0 && !fused_merge) {
    MergeFn mf = pick_merge(a->dtype, g.head_dim);
    hipLaunchKernelGGL(mf, dim3(a->batch * g.num_kv_heads, (gqa * g.head_dim / 4 + kBlock - 1) / kBlock), dim3(kBlock), 0,
                       st, a->unit_splits,
                       a->unit_partial_base, p.part_o, p.part_lse, a->out, a->lse, g.num_kv_heads, gqa);
    e = hipGetLastError();
    if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "merge launch failed: %s", hipGetErrorString(e));
  }
  return TG_OK;
}


}  // namespace

extern "C" {

size_t tg_decode_workspace_bytes(const tg_geometry* geom, int32_t batch, int32_t num_partials) {
  if (!geom || geom->num_kv_heads < 1 || geom->num_q_heads < geom->num_kv_heads || num_partials < 0 || batch < 0)
    return 0;
  const size_t gqa = (size_t)(geom->num_q_heads / geom->num_kv_heads);
  const size_t d = (size_t)geom->head_dim;
  // fp32 partial outputs, then their lse
  return align256((size_t)num_partials * gqa * d * sizeof(float)) +
         align256((size_t)num_partials * gqa * sizeof(float));
}

int32_t tg_decode_max_ctas(const tg_geometry* geom, int32_t dtype, int32_t device, int32_t* n_cta) {
  if (!n_cta) return tg::fail(TG_ERR_INVALID_ARG, "n_cta is NULL");
  if (int32_t rc = check_decode_shape(geom, dtype)) return rc;
  DecodeFn fn = pick_decode(dtype, geom->head_dim, geom->num_q_heads / geom->num_kv_heads);
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess)
    return tg::fail(TG_ERR_HIP, "hipDeviceGetAttribute failed for device %d", device);
  int prev = 0;
  if (hipGetDevice(&prev) != hipSuccess) return tg::fail(TG_ERR_HIP, "hipGetDevice failed");
  if (prev != device && hipSetDevice(device) != hipSuccess) return tg::fail(TG_ERR_HIP, "hipSetDevice failed");
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(fn), kBlock, 0);
  if (prev != device) (void)hipSetDevice(prev);
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "occupancy query failed: %s", hipGetErrorString(e));
  *n_cta = per_cu * cus * workers_per_wg(dtype, geom->head_dim, geom->num_q_heads / geom->num_kv_heads);
  return TG_OK;
}

int32_t tg_decode(const tg_decode_args* a, void* hip_stream) {
  if (!a) return tg::fail(TG_ERR_INVALID_ARG, "args is NULL");
  return decode_impl(a, a->workspace, a->workspace_bytes, hip_stream);
}

int32_t tg_decode_noalloc(const tg_decode_args* a, void* hip_stream) {
  if (!a) return tg::fail(TG_ERR_INVALID_ARG, "args is NULL");
  if (int32_t rc = check_decode_shape(&a->geom, a->dtype)) return rc;
  if (a->batch < 1 || a->num_partials < 0) return tg::fail(TG_ERR_INVALID_ARG, "batch must be >= 1, num_partials >= 0");
  const size_t need = tg_decode_workspace_bytes(&a->geom, a->batch, a->num_partials);
  if (need > (size_t)TG_DECODE_NOALLOC_MAX_BYTES - kScratchCounters)
    return tg::fail(TG_ERR_BUFFER_TOO_SMALL,
                    "tg_decode_noalloc: %d partials need %zu bytes of scratch, the static scratch holds %zu",
                    a->num_partials, need, (size_t)TG_DECODE_NOALLOC_MAX_BYTES - kScratchCounters);
  void* ws = nullptr;
  if (int32_t rc = scratch_address(&ws)) return rc;
  // the scratch starts with kScratchCounters bytes of merge arrival counters
  // (zero at load; every call leaves them zero), then the partials
  tg_decode_args b = *a;
  char* base = static_cast<char*>(ws);
  const bool counters_fit = (size_t)a->batch * a->geom.num_kv_heads * sizeof(int32_t) <= kScratchCounters;
  b.merge_counters = a->merge_counters && counters_fit ? reinterpret_cast<int32_t*>(base) : nullptr;
  return decode_impl(&b, base + kScratchCounters, (size_t)TG_DECODE_NOALLOC_MAX_BYTES - kScratchCounters, hip_stream);
}

}  // extern "C"
