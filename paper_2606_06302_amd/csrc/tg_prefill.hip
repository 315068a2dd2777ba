// Ragged chunked-prefill attention for gfx950 (MI355X), bf16 MFMA.
//
// Chunked prefill (Section 2.2.1 of arXiv 2606.06302) over Tangram's ragged
// compressed cache (Section 4.2): row i of request b's chunk, query head
// qh = h*gqa + j, attends to the kv_len[b][layer][h] retained history rows of
// KV head h (all visible) followed by chunk keys 0..i (causal, inclusive).
//
// Work decomposition.  The gqa query heads of a KV head are packed into the
// row dimension (row r = i*gqa + j), so every K/V tile is reused by gqa*rows
// queries.  One workgroup (4 waves) owns 128 consecutive rows of one (b, h);
// wave w owns 32 of them.  Key tiles of 32 keys: first the paged history (two
// pages per tile), then the chunk's own keys up to the workgroup's last row.
// Block ids are mapped XCD-aware: all row tiles of a (b, h) run on the same
// XCD (block id mod 8), so the history they share is read into one L2.
//
// Per key tile, each wave does (v_mfma_f32_32x32x16_bf16, fp32 accumulate):
//   S^T[key][row] = K Q^T   (A = K rows from LDS, B = Q rows in registers)
//   online softmax per row  (a lane owns one row: max over its 16 keys plus
//                            one permlane32 swap with the lane holding the rest)
//   O^T[dv][row] += V^T P^T (A = V^T from LDS, B = P^T straight from the
//                            lane's own S^T registers, rounded to bf16)
// The B layout of P^T requires the 32 keys of a tile in the order
// sigma(kappa) = 16*(kappa/16) + 8*((kappa%8)/4) + 4*((kappa%16)/8) + kappa%4,
// so V^T is written to LDS transposed in that order.
#include <hip/hip_runtime.h>

#include <cmath>

#include "tg_device.h"
#include "tg_internal.h"

namespace {

using namespace tgd;

typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kD = 128;          // head_dim
constexpr int kPage = 16;
constexpr int kWaves = 4;
constexpr int kBlock = 64 * kWaves;
constexpr int kRows = 32 * kWaves;   // query rows per workgroup
constexpr int kKeys = 32;            // keys per tile
constexpr int kKRow = kD * 2 + 16;   // LDS bytes per K row (padded)
constexpr int kVRow = kKeys * 2 + 16;   // LDS bytes per V^T row (padded)
constexpr int kKBytes = kKeys * kKRow;
constexpr int kVBytes = kD * kVRow;
constexpr int kBufBytes = kKBytes + kVBytes;
constexpr float kSlack = 8.0f;

struct PrefillParams {
  const uint16_t* q;        // [B][C][Hq][d]
  const uint16_t* k_new;    // [B][C][H][d]
  const uint16_t* v_new;
  const uint16_t* pool;     // [pages][2][Hp][P][d]
  const int32_t* pt_pages;
  const int64_t* pt_offsets;
  const int32_t* kv_len;    // [B][L][H]
  const int32_t* group_of;  // [L][H]
  const int32_t* slot_of;
  uint16_t* out;            // [B][C][Hq][d]
  int32_t batch, chunk, layer, num_layers, num_kv_heads, num_groups, heads_per_group, gqa;
  int32_t row_tiles;        // ceil(chunk*gqa / kRows)
  float scale_log2;
};

__device__ __forceinline__ f32x16 mfma(const u4& a, const u4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0,
                                                 0);
}

// kappa position (0..31) of key n (0..31) of a tile: inverse of sigma
__device__ __forceinline__ int kappa_of(int n) {
  const int ks = n >> 4, a = (n >> 3) & 1, hf = (n >> 2) & 1, b = n & 3;
  return ks * 16 + hf * 8 + a * 4 + b;
}

__global__ void __launch_bounds__(kBlock) tg_prefill_kernel(PrefillParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * kBufBytes];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tid = threadIdx.x;

  // XCD-aware block -> (unit, row tile): units round-robin over the 8 XCDs
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int unit = xcd + 8 * (local / p.row_tiles);
  const int rt = local % p.row_tiles;
  const int n_units = p.batch * p.num_kv_heads;
  if (unit >= n_units) return;
  const int b = unit / p.num_kv_heads, h = unit % p.num_kv_heads;
  const int C = p.chunk, gqa = p.gqa;
  const int Hq = p.num_kv_heads * gqa;
  const int rows_total = C * gqa;
  const int row0 = rt * kRows;
  const int hist = p.kv_len[((int64_t)b * p.num_layers + p.layer) * p.num_kv_heads + h];
  const int grp = p.group_of[(int64_t)p.layer * p.num_kv_heads + h];
  const int slot = p.slot_of[(int64_t)p.layer * p.num_kv_heads + h];
  const int64_t tbase = p.pt_offsets[((int64_t)b * p.num_layers + p.layer) * p.num_groups + grp];
  const int i_last = min(C - 1, (min(row0 + kRows, rows_total) - 1) / gqa);   // last chunk row of the block
  const int n_hist_tiles = (hist + kKeys - 1) / kKeys;
  const int n_tiles = n_hist_tiles + (i_last + kKeys) / kKeys;

  // this lane's query row (B operand of S^T and the row it owns in S^T / O^T)
  const int my_row = row0 + wave * 32 + (lane & 31);
  const bool row_ok = my_row < rows_total;
  const int my_i = row_ok ? my_row / gqa : 0;
  const int my_j = row_ok ? my_row % gqa : 0;
  const int wave_i_max = min(C - 1, (min(row0 + wave * 32 + 32, rows_total) - 1) / gqa);
  const int hf = lane >> 5;
  u4 qb[8];
  {
    const u4* qp = reinterpret_cast<const u4*>(p.q + (((int64_t)b * C + my_i) * Hq + h * gqa + my_j) * kD);
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) qb[kk] = row_ok ? qp[kk * 2 + hf] : u4(0u);
  }

  // K/V tile loaders: thread t fetches K chunks t and t+256 of the tile
  // (key = idx/16, chunk = idx%16) and V chunk t%16 of keys 2*(t/16), 2*(t/16)+1.
  auto key_src = [&](int tile, int n, int which) -> const u4* {   // nullptr if the key is masked out
    if (tile < n_hist_tiles) {
      const int t = tile * kKeys + n;
      if (t >= hist) return nullptr;
      const int64_t page = p.pt_pages[tbase + t / kPage];
      const uint16_t* base = p.pool + (((page * 2 + which) * p.heads_per_group + slot) * kPage + t % kPage) * kD;
      return reinterpret_cast<const u4*>(base);
    }
    const int c = (tile - n_hist_tiles) * kKeys + n;
    if (c >= C) return nullptr;
    const uint16_t* src = which == 0 ? p.k_new : p.v_new;
    return reinterpret_cast<const u4*>(src + (((int64_t)b * C + c) * p.num_kv_heads + h) * kD);
  };
  u4 kreg[2], vreg[2];
  auto load_tile = [&](int tile) {
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const int idx = tid + x * kBlock;
      const u4* src = key_src(tile, idx >> 4, 0);
      kreg[x] = src ? src[idx & 15] : u4(0u);
    }
    const int kp = tid >> 4, c = tid & 15;
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const u4* src = key_src(tile, 2 * kp + x, 1);
      vreg[x] = src ? src[c] : u4(0u);
    }
  };
  auto store_tile = [&](int buf) {
    unsigned char* kb = smem + buf * kBufBytes;
    unsigned char* vb = kb + kKBytes;
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const int idx = tid + x * kBlock;
      *reinterpret_cast<u4*>(kb + (idx >> 4) * kKRow + (idx & 15) * 16) = kreg[x];
    }
    // V^T: dword (v[n][d], v[n+1][d]) at row d, column kappa(n)/2
    const int kp = tid >> 4, c = tid & 15;
    const int col = kappa_of(2 * kp) >> 1;
    const uint32_t* v0 = reinterpret_cast<const uint32_t*>(&vreg[0]);
    const uint32_t* v1 = reinterpret_cast<const uint32_t*>(&vreg[1]);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t lo = __builtin_amdgcn_perm(v1[w], v0[w], 0x05040100u);
      const uint32_t hi = __builtin_amdgcn_perm(v1[w], v0[w], 0x07060302u);
      const int d = c * 8 + 2 * w;
      *reinterpret_cast<uint32_t*>(vb + d * kVRow + col * 4) = lo;
      *reinterpret_cast<uint32_t*>(vb + (d + 1) * kVRow + col * 4) = hi;
    }
  };

  f32x16 acc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) acc[t] = f32x16(0.f);
  float m = -INFINITY, l = 0.f;
  const float cs = p.scale_log2;

  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int tile = 0; tile < n_tiles; ++tile) {
    const int buf = tile & 1;
    const bool more = tile + 1 < n_tiles;
    if (more) load_tile(tile + 1);
    const unsigned char* kb = smem + buf * kBufBytes;
    const unsigned char* vb = kb + kKBytes;
    const bool is_chunk = tile >= n_hist_tiles;
    const int c0 = (tile - n_hist_tiles) * kKeys;   // first chunk key of the tile
    // skip a chunk tile that is entirely in the future of this wave's rows
    if (!(is_chunk && c0 > wave_i_max)) {
      f32x16 s = f32x16(0.f);
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const u4 a = *reinterpret_cast<const u4*>(kb + (lane & 31) * kKRow + (kk * 2 + hf) * 16);
        s = mfma(a, qb[kk], s);
      }
      // lane holds keys n(r) = 8*(r/4) + 4*hf + r%4 of its row
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = 8 * (r >> 2) + 4 * hf + (r & 3);
        bool ok;
        if (is_chunk) ok = c0 + n <= my_i && c0 + n < C;
        else ok = tile * kKeys + n < hist;
        s[r] = ok ? s[r] : -INFINITY;
        mx = fmaxf(mx, s[r]);
      }
      mx = swap32_max(mx);
      if ((mx - m) * cs > kSlack) {   // raise the running max (rare after the first tile)
        const float alpha = fast_exp2((m - mx) * cs);
        m = mx;
        l *= alpha;
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] *= alpha;
      }
      const float mcs = m * cs;
      uint32_t pw[8];
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const float p0 = fast_exp2(fmaf(s[r], cs, -mcs));
        const float p1 = fast_exp2(fmaf(s[r + 1], cs, -mcs));
        l += p0 + p1;
        pw[r >> 1] = uint32_t(f32_to_bf16(p0)) | (uint32_t(f32_to_bf16(p1)) << 16);
      }
      u4 pb0, pb1;
      pb0.x = pw[0]; pb0.y = pw[1]; pb0.z = pw[2]; pb0.w = pw[3];
      pb1.x = pw[4]; pb1.y = pw[5]; pb1.z = pw[6]; pb1.w = pw[7];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const unsigned char* vrow = vb + (t * 32 + (lane & 31)) * kVRow;
        acc[t] = mfma(*reinterpret_cast<const u4*>(vrow + hf * 16), pb0, acc[t]);
        acc[t] = mfma(*reinterpret_cast<const u4*>(vrow + 32 + hf * 16), pb1, acc[t]);
      }
    }
    if (more) store_tile(buf ^ 1);
    __syncthreads();
  }
  // row sum over both halves of the row, then O = O^T / l
  l = swap32_sum(l);
  if (!row_ok) return;
  const float inv = 1.f / l;
  uint16_t* orow = p.out + (((int64_t)b * C + my_i) * Hq + h * gqa + my_j) * kD;
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int dv = t * 32 + 8 * r4 + 4 * hf;
      uint32_t w0 = uint32_t(f32_to_bf16(acc[t][r4 * 4 + 0] * inv)) | (uint32_t(f32_to_bf16(acc[t][r4 * 4 + 1] * inv)) << 16);
      uint32_t w1 = uint32_t(f32_to_bf16(acc[t][r4 * 4 + 2] * inv)) | (uint32_t(f32_to_bf16(acc[t][r4 * 4 + 3] * inv)) << 16);
      *reinterpret_cast<uint2*>(orow + dv) = make_uint2(w0, w1);
    }
}

}  // namespace

extern "C" {

size_t tg_prefill_workspace_bytes(const tg_prefill_args* args) {
  (void)args;
  return 0;
}

int32_t tg_prefill(const tg_prefill_args* a, void* hip_stream) {
  if (!a) return tg::fail(TG_ERR_INVALID_ARG, "args is NULL");
  const tg_geometry& g = a->geom;
  if (int32_t rc = tg::check_geometry(&g)) return rc;
  if (a->dtype != TG_BF16) return tg::fail(TG_ERR_UNSUPPORTED, "prefill supports bf16 only");
  if (g.head_dim != kD) return tg::fail(TG_ERR_UNSUPPORTED, "prefill supports head_dim 128 only (got %d)", g.head_dim);
  if (g.page_size != kPage) return tg::fail(TG_ERR_UNSUPPORTED, "prefill supports page_size 16 only");
  const int gqa = g.num_q_heads / g.num_kv_heads;
  if (gqa < 1 || gqa > 16) return tg::fail(TG_ERR_UNSUPPORTED, "prefill supports 1..16 query heads per KV head");
  if (a->batch < 1 || a->chunk_len < 1 || a->layer < 0 || a->layer >= g.num_layers)
    return tg::fail(TG_ERR_INVALID_ARG, "batch and chunk_len must be >= 1, layer in range");
  if (!a->q || !a->k_new || !a->v_new || !a->kv_pool || !a->pt_pages || !a->pt_offsets || !a->kv_len ||
      !a->group_of || !a->slot_of || !a->out)
    return tg::fail(TG_ERR_INVALID_ARG, "NULL device pointer");
  PrefillParams p;
  p.q = static_cast<const uint16_t*>(a->q);
  p.k_new = static_cast<const uint16_t*>(a->k_new);
  p.v_new = static_cast<const uint16_t*>(a->v_new);
  p.pool = static_cast<const uint16_t*>(a->kv_pool);
  p.pt_pages = a->pt_pages;
  p.pt_offsets = a->pt_offsets;
  p.kv_len = a->kv_len;
  p.group_of = a->group_of;
  p.slot_of = a->slot_of;
  p.out = static_cast<uint16_t*>(a->out);
  p.batch = a->batch;
  p.chunk = a->chunk_len;
  p.layer = a->layer;
  p.num_layers = g.num_layers;
  p.num_kv_heads = g.num_kv_heads;
  p.num_groups = g.num_kv_heads / g.heads_per_group;
  p.heads_per_group = g.heads_per_group;
  p.gqa = gqa;
  p.row_tiles = (a->chunk_len * gqa + kRows - 1) / kRows;
  const float scale = a->sm_scale != 0.f ? a->sm_scale : 1.0f / std::sqrt((float)kD);
  p.scale_log2 = scale * kLog2e;
  const int units = a->batch * g.num_kv_heads;
  const int blocks = 8 * ((units + 7) / 8) * p.row_tiles;
  hipLaunchKernelGGL(tg_prefill_kernel, dim3(blocks), dim3(kBlock), 0, static_cast<hipStream_t>(hip_stream), p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "prefill launch failed: %s", hipGetErrorString(e));
  return TG_OK;
}

}  // extern "C"
