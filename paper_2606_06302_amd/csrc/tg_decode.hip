// Ragged paged split-KV decode attention for gfx950 (MI355X).
//
// One decode step of one layer over Tangram's ragged cache (Section 4.2 of
// arXiv 2606.06302): every KV head h of request b keeps its own number of
// retained rows, stored in the pages of its head group.  The host partition
// (tg_build_plan, Algorithm 1's proportional rule) cuts every (b, h) into
// page-aligned chunks and places them on n_bins persistent workgroups; the
// kernel below runs bin k on workgroup k.  Chunks of a split unit write fp32
// partial (o, lse) and tg_merge_kernel combines them with a log-sum-exp
// merge (split-KV decoding, Section 2.2.3).
//
// Kernel design (HBM-bound streaming, no MFMA):
//   * 4 waves per workgroup; the pages of an item are dealt round-robin to the
//     waves, each wave keeps its own online-softmax state, and the four states
//     are merged through LDS at the end of the item.
//   * A page slab (P=16 rows of one head, d*sizeof(T) bytes each) is read with
//     one 16-byte load per lane per 64 chunks, so every load instruction
//     touches whole contiguous 1 KiB runs of the slab.  Lane l owns chunk
//     l % CPR of token row l / CPR (CPR = 16-byte chunks per row).
//   * q.k uses v_dot2_f32_bf16 on the raw bf16 pairs (fp32 FMAs for fp32
//     data) and a DPP all-reduce over the CPR lanes of a row; the per-page
//     max uses the gfx950 permlane16/32 swaps across rows.
//   * Online softmax in base 2 with the scale folded into one FMA; the running
//     max only rescales the accumulators when it grows (wave-uniform branch).
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

struct alignas(16) u4 {
  uint32_t x, y, z, w;
};

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

// Geometry of the per-lane tiling for a given storage type and head_dim.
template <typename T, int D>
struct Tile {
  static constexpr int kRowBytes = D * Store<T>::kBytes;
  static constexpr int kCPR = kRowBytes / 16;    // 16-byte chunks per token row
  static constexpr int kEPC = 16 / Store<T>::kBytes;  // elements per chunk
  static constexpr int kTPL = 64 / kCPR;         // token rows per wave load
  static constexpr int kSlots = kPage / kTPL;    // loads per lane per page slab
  static constexpr int kSlabChunks = kPage * kCPR;  // 16-byte chunks per slab
  static_assert(kCPR == 8 || kCPR == 16 || kCPR == 32, "unsupported row size");
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
  void* out;
  float* lse;
  float* part_o;             // [num_partials][gqa][d]
  float* part_lse;           // [num_partials][gqa]
  int64_t page_chunks;       // 16-byte chunks per physical page
  int32_t heads_per_group;
  int32_t num_q_heads;
  float scale_log2;          // sm_scale * log2(e)
  float scale;               // sm_scale
};

template <typename T, int D, int GQA>
__global__ void __launch_bounds__(kBlock) tg_decode_kernel(DecodeParams p) {
  using TL = Tile<T, D>;
  constexpr int CPR = TL::kCPR, EPC = TL::kEPC, TPL = TL::kTPL, NS = TL::kSlots;

  __shared__ float sm_m[kWaves][GQA];
  __shared__ float sm_l[kWaves][GQA];
  __shared__ float sm_acc[kWaves][GQA][D];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int c = lane % CPR;       // chunk of the row this lane owns
  const int r = lane / CPR;       // token row within one wave load
  const int bin = blockIdx.x;
  const int it_begin = p.bin_offsets[bin], it_end = p.bin_offsets[bin + 1];
  const float cs = p.scale_log2;

  for (int it = it_begin; it < it_end; ++it) {
    const tg_work_item item = p.items[it];
    const int qh0 = item.kv_head * GQA;
    // q chunks of this lane for all GQA query heads
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
    const int32_t* pt = p.pt_pages + item.pt_base + item.tok_begin / kPage;
    const int64_t slab_k = (int64_t)item.slot * TL::kSlabChunks;
    const int64_t slab_v = ((int64_t)p.heads_per_group + item.slot) * TL::kSlabChunks;

    u4 kc[NS], vc[NS];
    auto load_page = [&](int pi, u4* kd, u4* vd) {
      const int64_t pg = (int64_t)pt[pi] * p.page_chunks;
      const u4* kb = p.pool + pg + slab_k + lane;
      const u4* vb = p.pool + pg + slab_v + lane;
#pragma unroll
      for (int j = 0; j < NS; ++j) {
        kd[j] = kb[j * 64];
        vd[j] = vb[j * 64];
      }
    };
    int pi = wave;
    if (pi < npages) load_page(pi, kc, vc);
    for (; pi < npages; pi += kWaves) {
      u4 kn[NS], vn[NS];
      const bool more = pi + kWaves < npages;
      if (more) load_page(pi + kWaves, kn, vn);
      const int nvalid = min(kPage, ntok - pi * kPage);  // rows of this page in range
      // logits s[j][g] for this lane's token rows
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
          if (!ok) vc[j] = u4{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int g = 0; g < GQA; ++g) {
        float mx = s[0][g];
#pragma unroll
        for (int j = 1; j < NS; ++j) mx = fmaxf(mx, s[j][g]);
        mx = rows_max<CPR>(mx);
        if (mx > m[g]) {   // uniform across the wave
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
      if (more) {
#pragma unroll
        for (int j = 0; j < NS; ++j) {
          kc[j] = kn[j];
          vc[j] = vn[j];
        }
      }
    }
    // combine the token rows of this wave, then the waves through LDS
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
    for (int o = threadIdx.x; o < GQA * D; o += kBlock) {
      const int g = o / D, e = o % D;
      float M = sm_m[0][g];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) M = fmaxf(M, sm_m[w][g]);
      float L = 0.f, A = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float f = fast_exp2((sm_m[w][g] - M) * cs);   // 0 for a wave with no rows
        L = fmaf(sm_l[w][g], f, L);
        A = fmaf(sm_acc[w][g][e], f, A);
      }
      const float O = A / L;
      const float lse_nat = M * p.scale + logf(L);
      if (item.out_idx < 0) {
        store_out<T>(static_cast<T*>(p.out) + ((int64_t)item.b * p.num_q_heads + qh0 + g) * D + e, O);
        if (p.lse && e == 0) p.lse[(int64_t)item.b * p.num_q_heads + qh0 + g] = lse_nat;
      } else {
        p.part_o[((int64_t)item.out_idx * GQA + g) * D + e] = O;
        if (e == 0) p.part_lse[(int64_t)item.out_idx * GQA + g] = lse_nat;
      }
    }
    __syncthreads();
  }
}

// Log-sum-exp merge of the split partials of every unit (b, h) with more
// than one split: lse* = log sum_i e^{lse_i}, O = sum_i e^{lse_i - lse*} o_i.
template <typename T, int D>
__global__ void __launch_bounds__(kBlock) tg_merge_kernel(const int32_t* unit_splits, const int32_t* unit_base,
                                                         const float* part_o, const float* part_lse, void* out,
                                                         float* lse, int32_t num_kv_heads, int32_t gqa) {
  const int u = blockIdx.x;
  const int s = unit_splits[u];
  if (s <= 1) return;
  const int base = unit_base[u];
  const int b = u / num_kv_heads, h = u % num_kv_heads;
  const int hq = num_kv_heads * gqa;
  for (int o = threadIdx.x; o < gqa * D; o += kBlock) {
    const int g = o / D, e = o % D;
    float M = -INFINITY;
    for (int i = 0; i < s; ++i) M = fmaxf(M, part_lse[(int64_t)(base + i) * gqa + g]);
    float L = 0.f, A = 0.f;
    for (int i = 0; i < s; ++i) {
      const float w = __expf(part_lse[(int64_t)(base + i) * gqa + g] - M);
      L += w;
      A = fmaf(w, part_o[((int64_t)(base + i) * gqa + g) * D + e], A);
    }
    const int64_t row = (int64_t)b * hq + h * gqa + g;
    store_out<T>(static_cast<T*>(out) + row * D + e, A / L);
    if (lse && e == 0) lse[row] = M + logf(L);
  }
}

using DecodeFn = void (*)(DecodeParams);
using MergeFn = void (*)(const int32_t*, const int32_t*, const float*, const float*, void*, float*, int32_t, int32_t);

template <typename T, int D, int... G>
constexpr auto make_decode_table(std::integer_sequence<int, G...>) {
  return std::array<DecodeFn, sizeof...(G)>{&tg_decode_kernel<T, D, G + 1>...};
}

constexpr int kMaxGqa = 16;
// [dtype][d == 128][gqa - 1]
const std::array<DecodeFn, kMaxGqa> kDecodeF32D64 = make_decode_table<float, 64>(std::make_integer_sequence<int, kMaxGqa>{});
const std::array<DecodeFn, kMaxGqa> kDecodeF32D128 = make_decode_table<float, 128>(std::make_integer_sequence<int, kMaxGqa>{});
const std::array<DecodeFn, kMaxGqa> kDecodeBF16D64 = make_decode_table<uint16_t, 64>(std::make_integer_sequence<int, kMaxGqa>{});
const std::array<DecodeFn, kMaxGqa> kDecodeBF16D128 = make_decode_table<uint16_t, 128>(std::make_integer_sequence<int, kMaxGqa>{});

DecodeFn pick_decode(int dtype, int d, int gqa) {
  if (gqa < 1 || gqa > kMaxGqa) return nullptr;
  if (dtype == TG_F32 && d == 64) return kDecodeF32D64[gqa - 1];
  if (dtype == TG_F32 && d == 128) return kDecodeF32D128[gqa - 1];
  if (dtype == TG_BF16 && d == 64) return kDecodeBF16D64[gqa - 1];
  if (dtype == TG_BF16 && d == 128) return kDecodeBF16D128[gqa - 1];
  return nullptr;
}

MergeFn pick_merge(int dtype, int d) {
  if (dtype == TG_F32 && d == 64) return &tg_merge_kernel<float, 64>;
  if (dtype == TG_F32 && d == 128) return &tg_merge_kernel<float, 128>;
  if (dtype == TG_BF16 && d == 64) return &tg_merge_kernel<uint16_t, 64>;
  if (dtype == TG_BF16 && d == 128) return &tg_merge_kernel<uint16_t, 128>;
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
  // partial outputs, partial lse, then one int32 counter per (b, h) unit
  return align256((size_t)num_partials * gqa * d * sizeof(float)) +
         align256((size_t)num_partials * gqa * sizeof(float)) +
         align256((size_t)batch * geom->num_kv_heads * sizeof(int32_t));
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
  DecodeParams p;
  p.q = a->q;
  p.pool = static_cast<const u4*>(a->kv_pool);
  p.pt_pages = a->pt_pages;
  p.items = a->items;
  p.bin_offsets = a->bin_offsets;
  p.out = a->out;
  p.lse = a->lse;
  p.part_o = static_cast<float*>(a->workspace);
  p.part_lse = a->workspace ? reinterpret_cast<float*>(static_cast<char*>(a->workspace) +
                                                       align256((size_t)a->num_partials * gqa * g.head_dim * 4))
                            : nullptr;
  p.page_chunks = (int64_t)g.heads_per_group * 2 * kPage * g.head_dim * esz / 16;
  p.heads_per_group = g.heads_per_group;
  p.num_q_heads = g.num_q_heads;
  p.scale = a->sm_scale != 0.f ? a->sm_scale : 1.0f / std::sqrt((float)g.head_dim);
  p.scale_log2 = p.scale * kLog2e;
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  if (a->num_items > 0) {
    DecodeFn fn = pick_decode(a->dtype, g.head_dim, gqa);
    hipLaunchKernelGGL(fn, dim3(a->n_bins), dim3(kBlock), 0, st, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "decode launch failed: %s", hipGetErrorString(e));
  }
  if (a->num_partials > 0) {
    MergeFn mf = pick_merge(a->dtype, g.head_dim);
    hipLaunchKernelGGL(mf, dim3(a->batch * g.num_kv_heads), dim3(kBlock), 0, st, a->unit_splits,
                       a->unit_partial_base, p.part_o, p.part_lse, a->out, a->lse, g.num_kv_heads, gqa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "merge launch failed: %s", hipGetErrorString(e));
  }
  return TG_OK;
}

}  // extern "C"
