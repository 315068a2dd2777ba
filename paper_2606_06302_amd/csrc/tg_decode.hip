// Ragged paged split-KV decode attention for gfx950 (MI355X).
//
// One decode step of one layer over Tangram's ragged cache (Section 4.2 of
// arXiv 2606.06302): every KV head h of request b keeps its own number of
// retained rows, stored in the pages of its head group.  The host partition
// (tg_build_plan, Algorithm 1's proportional rule) cuts every (b, h) into
// page-aligned chunks and places them on n_bins persistent workgroups; the
// kernel runs bin k on workgroup k.  A chunk of a split unit writes an fp32
// partial (o, lse) and tg_merge_kernel, launched right after on the same
// stream, combines the partials of every split unit with a log-sum-exp merge
// (split-KV decoding, Section 2.2.3).  The merge is a separate launch on
// purpose: making one workgroup's partials visible to another inside a launch
// needs agent-scope fences, which on MI355X write back and invalidate the
// whole L2 of an XCD and cost more than half of the kernel's bandwidth.
//
// Both kernels deal the pages of an item round-robin to the 4 waves of the
// workgroup; every wave keeps its own online-softmax state and the states are
// merged through LDS at the end of the item.  The wave index is made
// wave-uniform (readfirstlane) so that all item/page bookkeeping is scalar.
#include <hip/hip_runtime.h>

#include <array>
#include <cmath>
#include <cstring>
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
  float scale_log2;          // sm_scale * log2(e)
  float scale;               // sm_scale
};

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

  for (int it = it_begin; it < it_end; ++it) {
    const tg_work_item item = items[it];
    const int qh0 = item.kv_head * GQA;
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
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Fast path for bf16, head_dim 128 and G = gqa in {4, 8, 16}.
//
// A wave works on a step of SP consecutive pages of an item (SP*16 tokens).
// Steps of an item are dealt round-robin to the 4 waves.  Each wave streams
// its steps through registers into its own LDS buffers: while step n is
// computed from LDS, step n+1 (SP*8 KiB) is already in flight into the
// staging registers - one unconditional issue per step, so the loads land
// directly in the loop-carried registers and are only waited for when they
// are written to LDS one iteration later.  Page ids are read with vector
// loads (kept off the LDS/scalar counter) one step ahead of their use.
//   * q.k: lane (h = lane % G, row = lane / G) holds the whole 128-dim query of
//     head h and computes complete dot products for tokens row, row + 64/G, ...
//     of the step (no cross-lane reduction).  K slabs are stored in LDS with
//     chunk c of token row r at position c ^ r, so the 64/G tokens read in one
//     instruction hit distinct banks while lanes of one token broadcast.
//   * p.v: lane owns dims (2*lane, 2*lane+1) of all G heads; V rows of two
//     tokens are interleaved with v_perm_b32 and p is rounded to bf16 pairs, so
//     each v_dot2_f32_bf16 accumulates two tokens at once (fp32 accumulate).
//   * The running max of a head is only raised when a step exceeds it by more
//     than 8 (in log2 units), so accumulator rescales are rare; p stays <= 2^8.
template <int SP>
struct Stage {
  u4 k[4 * SP], v[4 * SP];
};

// Loads the K and V slabs of `slot` in pages pg[0..SP): lane l takes 16-byte
// chunks l, l+64, l+128, l+192 of every slab.
template <int SP>
__device__ __forceinline__ Stage<SP> fetch_step(const DecodeParams& p, const u4* __restrict__ pool,
                                                const int64_t (&pg)[SP], int slot, int lane) {
  Stage<SP> s;
#pragma unroll
  for (int q = 0; q < SP; ++q) {
    const u4* base = pool + pg[q] * p.page_chunks;
    const u4* kb = base + slot * 256 + lane;
    const u4* vb = base + (p.heads_per_group + slot) * 256 + lane;
#pragma unroll
    for (int j = 0; j < 4; ++j) {   // streamed once: non-temporal
      s.k[q * 4 + j] = __builtin_nontemporal_load(kb + j * 64);
      s.v[q * 4 + j] = __builtin_nontemporal_load(vb + j * 64);
    }
  }
  return s;
}

template <int G, int SP>
__global__ void __launch_bounds__(kBlock) tg_decode_fast_kernel(DecodeParams p, const tg_work_item* __restrict__ items,
                                                               const int32_t* pt_pages,
                                                               const int32_t* __restrict__ bin_offsets,
                                                               const u4* __restrict__ pool) {
  constexpr int D = 128;
  constexpr int kTok = SP * kPage;     // tokens per step
  constexpr int TR = 64 / G;           // token rows per q.k pass
  constexpr int TPL = kTok / TR;       // tokens per lane in q.k
  constexpr float kSlack = 8.0f;
  constexpr int kBufU4 = SP * 512;     // 16-byte slots of one wave's K+V buffer
  constexpr int kAccStride = kBufU4 * 4;
  static_assert(G == 4 || G == 8 || G == 16, "fast path covers gqa 4, 8, 16");
  static_assert(G * D <= kAccStride, "accumulators must fit the wave's buffer");

  // per wave: SP swizzled K slabs then SP V slabs; the end-of-item merge reuses them
  __shared__ u4 sm_kv[kWaves][kBufU4];
  __shared__ uint32_t sm_p[kWaves][kTok / 2][G];
  __shared__ float sm_alpha[kWaves][G];
  __shared__ float sm_m[kWaves][G];
  __shared__ float sm_l[kWaves][G];

  const int lane = threadIdx.x & 63;
  const int wave = wave_id();
  const int h = lane % G;
  const int tr = lane / G;
  const int it_begin = bin_offsets[blockIdx.x], it_end = bin_offsets[blockIdx.x + 1];
  if (it_begin >= it_end) return;
  const float cs = p.scale_log2;
  u4* const kbuf = &sm_kv[wave][0];
  uint32_t* const vbuf = reinterpret_cast<uint32_t*>(&sm_kv[wave][SP * 256]);
  uint16_t* const pbuf16 = reinterpret_cast<uint16_t*>(&sm_p[wave][0][0]);

  // This wave's steps in processing order: steps wave, wave+4, ... of every
  // item of the bin.  The cursor caches its item's step/page counts, table
  // base and slot, so items are only read when the cursor enters a new item.
  struct Cursor {
    int it, si, ns, np, slot;
    int64_t base;   // index into pt_pages of the item's first page
  };
  auto enter = [&](Cursor& cu, int it) {
    const tg_work_item& im = items[it];
    cu.it = it;
    cu.si = wave;
    cu.np = (im.tok_end - im.tok_begin + kPage - 1) / kPage;
    cu.ns = (cu.np + SP - 1) / SP;
    cu.slot = im.slot;
    cu.base = im.pt_base + im.tok_begin / kPage;
  };
  // moves to the next step of this wave; returns false (cursor unchanged) at the end
  auto advance = [&](Cursor& cu) {
    if (cu.si + kWaves < cu.ns) {
      cu.si += kWaves;
      return true;
    }
    for (int j = cu.it + 1; j < it_end; ++j) {
      Cursor t;
      enter(t, j);
      if (t.ns > wave) {
        cu = t;
        return true;
      }
    }
    return false;
  };
  // Page ids of a step, read with a lane-varying address so the value stays in a
  // VGPR (lane q holds page q of the step) and is only waited for when
  // ids_of() extracts it one iteration later.  Pages past the item's end
  // repeat its last page (their rows are masked).
  auto load_ids = [&](const Cursor& cu) {
    return pt_pages[cu.base + min(cu.si * SP + (lane & (SP - 1)), cu.np - 1)];
  };
  auto ids_of = [&](int ids, int64_t (&pg)[SP]) {
#pragma unroll
    for (int q = 0; q < SP; ++q) pg[q] = __builtin_amdgcn_readlane(ids, q);
  };
  // c: step whose data is in flight into `st`; n: the step after it, whose page
  // ids are in flight into n_ids.  Past the end n repeats the last step (a
  // harmless reload).
  Cursor c;
  enter(c, it_begin);
  if (c.ns <= wave && !advance(c)) c.si = 0;   // a wave without steps loads one it never uses
  Cursor n = c;
  advance(n);
  int n_ids = load_ids(n);
  Stage<SP> st;
  {
    int64_t pg[SP];
    ids_of(load_ids(c), pg);
    st = fetch_step<SP>(p, pool, pg, c.slot, lane);
  }

  for (int it = it_begin; it < it_end; ++it) {
    const tg_work_item item = items[it];
    const int qrow = item.kv_head * G + h;
    u4 qv[16];
    {
      const u4* qb = reinterpret_cast<const u4*>(static_cast<const uint16_t*>(p.q) +
                                                 ((int64_t)item.b * p.num_q_heads + qrow) * D);
#pragma unroll
      for (int c = 0; c < 16; ++c) qv[c] = qb[c];
    }
    float m = -INFINITY, l = 0.f;
    float acc[G][2];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g][0] = acc[g][1] = 0.f;
    const int ntok = item.tok_end - item.tok_begin;
    const int ns = (ntok + kTok - 1) / kTok;

    for (int si = wave; si < ns; si += kWaves) {
      // staging registers -> LDS
#pragma unroll
      for (int q = 0; q < SP; ++q)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int ci = j * 64 + lane;
          const int r = ci >> 4, cc = ci & 15;
          kbuf[q * 256 + r * 16 + (cc ^ r)] = st.k[q * 4 + j];
          reinterpret_cast<u4*>(vbuf)[q * 256 + ci] = st.v[q * 4 + j];
        }
      // the next step of this wave (possibly in a later item) goes in flight;
      // the cursor moves first, so item reads never wait on page data
      {
        Cursor nn = n;
        advance(nn);
        const int nn_ids = load_ids(nn);
        int64_t pg[SP];
        ids_of(n_ids, pg);
        st = fetch_step<SP>(p, pool, pg, n.slot, lane);
        n = nn;
        n_ids = nn_ids;
      }

      const int nvalid = min(kTok, ntok - si * kTok);
      float s[TPL];
#pragma unroll
      for (int k = 0; k < TPL; ++k) {
        const int t = tr + k * TR;
        const int q = t >> 4, r = t & 15;
        float a = 0.f;
#pragma unroll
        for (int cc = 0; cc < 16; ++cc) a = chunk_dot<uint16_t>(kbuf[q * 256 + r * 16 + (cc ^ r)], qv[cc], a);
        s[k] = t < nvalid ? a : -INFINITY;
      }
      float mx = s[0];
#pragma unroll
      for (int k = 1; k < TPL; ++k) mx = fmaxf(mx, s[k]);
      if constexpr (G == 4) {
        mx = fmaxf(mx, dpp<0x124>(mx));   // row_ror:4
        mx = fmaxf(mx, dpp<kRowRor8>(mx));
      } else if constexpr (G == 8) {
        mx = fmaxf(mx, dpp<kRowRor8>(mx));
      }
      mx = swap32_max(swap16_max(mx));
      const bool raise = (mx - m) * cs > kSlack;
      if (__any(raise)) {
        const float m_new = raise ? mx : m;
        const float alpha = fast_exp2((m - m_new) * cs);   // 0 when m was -inf
        l *= alpha;
        m = m_new;
        if (tr == 0) sm_alpha[wave][h] = alpha;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const float a = sm_alpha[wave][g];
          acc[g][0] *= a;
          acc[g][1] *= a;
        }
      }
      const float mcs = m * cs;
#pragma unroll
      for (int k = 0; k < TPL; ++k) {
        const int t = tr + k * TR;
        const float pk = fast_exp2(fmaf(s[k], cs, -mcs));
        l += pk;
        pbuf16[((t >> 1) * G + h) * 2 + (t & 1)] = f32_to_bf16(pk);
      }
      const bool partial = nvalid < kTok;
#pragma unroll
      for (int pr = 0; pr < kTok / 2; ++pr) {
        const int t0 = 2 * pr, t1 = 2 * pr + 1;
        uint32_t v0 = vbuf[(t0 >> 4) * 1024 + (t0 & 15) * 64 + lane];
        uint32_t v1 = vbuf[(t1 >> 4) * 1024 + (t1 & 15) * 64 + lane];
        if (partial) {   // rows past the retained length may hold anything
          if (t0 >= nvalid) v0 = 0u;
          if (t1 >= nvalid) v1 = 0u;
        }
        const uint32_t lo = __builtin_amdgcn_perm(v1, v0, 0x05040100u);
        const uint32_t hi = __builtin_amdgcn_perm(v1, v0, 0x07060302u);
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const uint32_t pp = sm_p[wave][pr][g];
          acc[g][0] = dot2_bf16(pp, lo, acc[g][0]);
          acc[g][1] = dot2_bf16(pp, hi, acc[g][1]);
        }
      }
    }
    // this wave's state -> LDS (its own K/V buffer holds its accumulators)
    if constexpr (G == 4) {
      l += dpp<0x124>(l);
      l += dpp<kRowRor8>(l);
    } else if constexpr (G == 8) {
      l += dpp<kRowRor8>(l);
    }
    l = swap32_sum(swap16_sum(l));
    if (tr == 0) {
      sm_m[wave][h] = m;
      sm_l[wave][h] = l;
    }
    float* accw = reinterpret_cast<float*>(&sm_kv[wave][0]);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      accw[g * D + 2 * lane] = acc[g][0];
      accw[g * D + 2 * lane + 1] = acc[g][1];
    }
    __syncthreads();
    finish_item<uint16_t, G, D>(p, item, sm_m, sm_l, reinterpret_cast<const float*>(&sm_kv[0][0]), kAccStride);
    __syncthreads();
  }
}

constexpr int kFastStep = 2;   // pages per wave step in the fast path

// Log-sum-exp merge of the split partials of every unit (b, h) with more than
// one split: lse* = log sum_i e^{lse_i}, O = sum_i e^{lse_i - lse*} o_i.
// Grid (units, ceil(gqa*D / 256)): each thread owns one output element and
// makes a single pass with a running max, so the loads of consecutive splits
// are independent and issue back to back.
template <typename T, int D>
__global__ void __launch_bounds__(kBlock) tg_merge_kernel(const int32_t* __restrict__ unit_splits,
                                                         const int32_t* __restrict__ unit_base,
                                                         const float* __restrict__ part_o,
                                                         const float* __restrict__ part_lse, void* out, float* lse,
                                                         int32_t num_kv_heads, int32_t gqa) {
  const int u = blockIdx.x;
  const int s = unit_splits[u];
  const int o = blockIdx.y * kBlock + threadIdx.x;
  if (s <= 1 || o >= gqa * D) return;
  const int base = unit_base[u];
  const int b = u / num_kv_heads, h = u % num_kv_heads;
  const int64_t row0 = (int64_t)b * num_kv_heads * gqa + (int64_t)h * gqa;
  const int g = o / D, e = o % D;
  const float* pl = part_lse + (int64_t)base * gqa + g;
  const float* po = part_o + ((int64_t)base * gqa + g) * D + e;
  float m = -INFINITY, L = 0.f, A = 0.f;
#pragma unroll 8
  for (int i = 0; i < s; ++i) {
    const float li = pl[(int64_t)i * gqa];
    const float oi = po[(int64_t)i * gqa * D];
    const float mn = fmaxf(m, li);
    const float a = __expf(m - mn), w = __expf(li - mn);
    L = fmaf(L, a, w);
    A = fmaf(A, a, w * oi);
    m = mn;
  }
  store_out<T>(static_cast<T*>(out) + (row0 + g) * D + e, A / L);
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
const std::array<DecodeFn, kMaxGqa> kDecodeBF16D128 = make_decode_table<uint16_t, 128>(std::make_integer_sequence<int, kMaxGqa>{});

DecodeFn pick_decode(int dtype, int d, int gqa) {
  if (gqa < 1 || gqa > kMaxGqa) return nullptr;
  if (dtype == TG_BF16 && d == 128) {
    if (gqa == 4) return &tg_decode_fast_kernel<4, kFastStep>;
    if (gqa == 8) return &tg_decode_fast_kernel<8, kFastStep>;
    if (gqa == 16) return &tg_decode_fast_kernel<16, kFastStep>;
  }
  if (dtype == TG_F32 && d == 64) return kDecodeF32D64[gqa - 1];
  if (dtype == TG_F32 && d == 128) return kDecodeF32D128[gqa - 1];
  if (dtype == TG_BF16 && d == 64) return kDecodeBF16D64[gqa - 1];
  if (dtype == TG_BF16 && d == 128) return kDecodeBF16D128[gqa - 1];
  return nullptr;
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
  *n_cta = per_cu * cus;
  return TG_OK;
}

int32_t tg_decode(const tg_decode_args* a, void* hip_stream) {
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
  if (a->num_partials > 0 && (!a->workspace || a->workspace_bytes < need))
    return tg::fail(TG_ERR_BUFFER_TOO_SMALL, "workspace holds %zu bytes, need %zu", a->workspace_bytes, need);
  const int gqa = g.num_q_heads / g.num_kv_heads;
  const int esz = a->dtype == TG_F32 ? 4 : 2;
  const size_t o_bytes = align256((size_t)a->num_partials * gqa * g.head_dim * 4);
  char* ws = static_cast<char*>(a->workspace);
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
  p.scale = a->sm_scale != 0.f ? a->sm_scale : 1.0f / std::sqrt((float)g.head_dim);
  p.scale_log2 = p.scale * kLog2e;
  if (a->num_items == 0) return TG_OK;
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  DecodeFn fn = pick_decode(a->dtype, g.head_dim, gqa);
  hipLaunchKernelGGL(fn, dim3(a->n_bins), dim3(kBlock), 0, st, p, a->items, a->pt_pages, a->bin_offsets, p.pool);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "decode launch failed: %s", hipGetErrorString(e));
  if (a->num_partials > 0) {
    MergeFn mf = pick_merge(a->dtype, g.head_dim);
    hipLaunchKernelGGL(mf, dim3(a->batch * g.num_kv_heads, (gqa * g.head_dim + kBlock - 1) / kBlock), dim3(kBlock), 0,
                       st, a->unit_splits,
                       a->unit_partial_base, p.part_o, p.part_lse, a->out, a->lse, g.num_kv_heads, gqa);
    e = hipGetLastError();
    if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "merge launch failed: %s", hipGetErrorString(e));
  }
  return TG_OK;
}

}  // extern "C"
