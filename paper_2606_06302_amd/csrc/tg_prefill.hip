// Ragged chunked-prefill attention for gfx950 (MI355X), bf16 MFMA.
//
// Chunked prefill (Section 2.2.1 of arXiv 2606.06302) over Tangram's ragged
// compressed cache (Section 4.2): row i of request b's chunk, query head
// qh = h*gqa + j, attends to the kv_len[b][layer][h] retained history rows of
// KV head h (all visible) followed by chunk keys 0..i (causal, inclusive).
//
// Work decomposition.  The gqa query heads of a KV head are packed into the
// row dimension (row r = i*gqa + j), so every K/V tile is reused by gqa*rows
// queries.  One workgroup (8 waves, two per SIMD) owns 256 consecutive rows
// of one (b, h); wave w owns 32 of them (one 32-row MFMA column block).  With
// two waves per SIMD the matrix core runs one wave's products while the other
// does its softmax.  Key tiles of 64 keys:
// first the paged history (four pages per tile), then the chunk's own keys up
// to the workgroup's last row.  Blocks are placed XCD-aware: all row tiles of
// a (b, h) run on the same XCD (block id mod 8), so the history they share is
// read into one L2; the host schedule (tg_prefill_schedule) balances the units
// over the XCDs by their tile counts and starts the longest blocks first.
//
// Data movement.  Tiles stream into a 4-deep LDS ring with gfx950's
// global_load_lds_dwordx4 (no staging registers); wave w fetches key rows
// 8w..8w+7 of a tile (half a page of history).  The DMA is issued from inline
// assembly (invisible to the compiler's wait-count pass), every wave waits for
// its own part with an explicit vmcnt, and one barrier per tile then makes the
// whole tile visible and retires every read of the slot the next DMA refills.
// Page ids and table entries are read with scalar loads.
//
// Per 32-key block and 32-row column block (v_mfma_f32_32x32x16_bf16, fp32
// accumulate):
//   S^T[key][row] = K Q^T   (A = K rows from LDS, B = Q rows in registers)
//   online softmax per row  (a lane owns one row: max over its 16 keys plus
//                            one permlane32 swap with the lane holding the rest)
//   O^T[dv][row] += V^T P^T (B = P^T straight from the lane's own S^T
//                            registers, rounded to bf16; A = V^T read from the
//                            row-major V tile with ds_read_b64_tr_b16)
// The lane in half hf = lane / 32 holds S^T keys {4hf..4hf+3, 8+4hf..8+4hf+3}
// of each 16-key half block and feeds them as B's 8 k-indices, so the A
// operand takes the same keys: two transposed reads of 4 consecutive keys.
// V rows of the last history tile past the retained length are zeroed in LDS
// by the wave that fetched them, so the PV loop needs no mask.
// LDS layout: chunk c (16 bytes) of key row r sits at position c ^ (r mod 16)
// in the K tile and c ^ 4(r mod 4) in the V tile, so the K operand reads and
// the transposed V reads are bank-conflict free.
#include <hip/hip_runtime.h>

#include <cmath>

#include "tg_device.h"
#include "tg_internal.h"

namespace {

using namespace tgd;

typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_vs __attribute__((__vector_size__(4 * sizeof(__bf16))));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

#define TG_CONST __attribute__((address_space(4)))
#define TG_LDS __attribute__((address_space(3)))

constexpr int kPage = 16;
constexpr int kWaves = 8;
constexpr int kBlock = 64 * kWaves;
constexpr int kCB = 1;                         // 32-row MFMA column blocks per wave
constexpr int kRowsPerWave = 32 * kCB;
constexpr int kRows = kRowsPerWave * kWaves;   // query rows per workgroup
constexpr int kTile = 64;                      // keys per tile = 4 pages
static_assert(kRows == TG_PREFILL_ROWS && kTile == TG_PREFILL_TILE, "tg_prefill_schedule costs these tiles");
constexpr int kRing = 4;                       // LDS tile buffers
static_assert(kRing >= 2 && kRing <= 4, "the wait below covers up to two tiles in flight after the current one");
constexpr int kDmaRows = kTile / kWaves;       // key rows each wave fetches per tile
constexpr float kSlack = 8.0f;

// Shape constants of the kernel for head_dim D (64 or 128).  A key row is
// 2*D bytes = kChunks 16-byte chunks; one 1 KiB DMA instruction (64 lanes x
// 16 bytes) moves kRowsPerDma rows.  LDS swizzles: chunk c of key row r of a
// tile sits at position c ^ k_swz(r) in the K tile and c ^ v_swz(r) in the V
// tile (r taken mod 16, which is also the row within its page), chosen so
// that the q.k operand reads and the transposed V reads are bank-conflict free.
template <int D>
struct Shape {
  static_assert(D == 64 || D == 128, "head_dim 64 or 128");
  static constexpr int kChunks = D / 8;
  static constexpr int kRowsPerDma = 64 / kChunks;
  static constexpr int kDmaInst = kDmaRows / kRowsPerDma;   // 1 KiB instructions per K or V slab and wave
  static constexpr int kDmaPerTile = 2 * kDmaInst;
  static constexpr int kTileBytes = 2 * kTile * D * 2;      // K + V
  static constexpr int kK = D / 16;                         // 16-deep k steps of q.k
  static constexpr int kDB = D / 32;                        // 32-dim blocks of the output
  __device__ static constexpr int k_swz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
  __device__ static constexpr int v_swz(int r) { return D == 128 ? 4 * (r & 3) : 2 * (r & 3); }
};

struct PrefillParams {
  const uint16_t* q;        // [B][C][Hq][d]
  const u4* k_new;          // [B][C][H][d]
  const u4* v_new;
  const u4* pool;           // [pages][2][Hp][P][d]
  const int32_t* pt_pages;
  const int64_t* pt_offsets;
  const int32_t* kv_len;    // [B][L][H]
  const int32_t* group_of;  // [L][H]
  const int32_t* slot_of;
  uint16_t* out;            // [B][C][Hq][d]
  const int32_t* block_order;   // [gridDim.x] (unit * row_tiles + row tile) or -1, or NULL
  int32_t batch, chunk, layer, num_layers, num_kv_heads, num_groups, heads_per_group, gqa;
  int32_t row_tiles;        // ceil(chunk*gqa / kRows)
  float scale_log2;
};

__device__ __forceinline__ f32x16 mfma(const u4& a, const u4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0,
                                                 0);
}

__device__ __forceinline__ uint32_t lds_address(const void* ptr) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const TG_LDS void*)ptr));
}

// 16 bytes per lane from global memory into LDS at m0_base + 16 * lane.
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t m0_base) {
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(m0_base) : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ void barrier() { asm volatile("s_barrier" ::: "memory"); }

// (lo, hi) rounded to bf16 and packed into one dword (one v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2v));
}

// Lane l of each 16-lane block receives element l % 4 of the 8-byte rows
// addressed by lanes l/4, l/4 + 4, l/4 + 8, l/4 + 12 of the block.
__device__ __forceinline__ u2v lds_read_tr16(const void* ptr) {
  return __builtin_bit_cast(u2v, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((TG_LDS bf16x4_vs*)ptr));
}

template <int D>
__global__ void __launch_bounds__(kBlock) tg_prefill_kernel(PrefillParams p) {
  using S = Shape<D>;
  constexpr int kChunks = S::kChunks, kDmaInst = S::kDmaInst, kDmaPerTile = S::kDmaPerTile;
  constexpr int kTileBytes = S::kTileBytes, kRowsPerDma = S::kRowsPerDma;
  __shared__ u4 ring[kRing][2][kTile * kChunks];   // [slot][K, V][key row * kChunks + chunk position]

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

  // block -> (unit, row tile): the host schedule, or units round-robin over
  // the 8 XCDs (all row tiles of a unit on one XCD either way)
  const int n_units = p.batch * p.num_kv_heads;
  int unit, rt;
  if (p.block_order) {
    const int code = ((const TG_CONST int32_t*)p.block_order)[blockIdx.x];
    if (code < 0 || code >= n_units * p.row_tiles) return;
    unit = code / p.row_tiles;
    rt = code % p.row_tiles;
  } else {
    const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
    unit = xcd + 8 * (local / p.row_tiles);
    rt = local % p.row_tiles;
    if (unit >= n_units) return;
  }
  const int b = unit / p.num_kv_heads, h = unit % p.num_kv_heads;
  const int C = p.chunk, gqa = p.gqa;
  const int Hq = p.num_kv_heads * gqa;
  const int rows_total = C * gqa;
  const int row0 = rt * kRows;

  const TG_CONST int32_t* kv_len = (const TG_CONST int32_t*)p.kv_len;
  const TG_CONST int32_t* group_of = (const TG_CONST int32_t*)p.group_of;
  const TG_CONST int32_t* slot_of = (const TG_CONST int32_t*)p.slot_of;
  const TG_CONST int64_t* pt_offsets = (const TG_CONST int64_t*)p.pt_offsets;
  const TG_CONST int32_t* pt_pages = (const TG_CONST int32_t*)p.pt_pages;

  const int grp = group_of[(int64_t)p.layer * p.num_kv_heads + h];
  const int slot = slot_of[(int64_t)p.layer * p.num_kv_heads + h];
  const int64_t tidx = ((int64_t)b * p.num_layers + p.layer) * p.num_groups + grp;
  const int64_t tbase = pt_offsets[tidx];
  // the history is clamped to the head's table: [0, pages * page_size]
  const int64_t cap = (pt_offsets[tidx + 1] - tbase) * kPage;
  const int hist = (int)max<int64_t>(0, min<int64_t>(kv_len[((int64_t)b * p.num_layers + p.layer) * p.num_kv_heads + h], cap));
  const int npages = (hist + kPage - 1) / kPage;
  const int i_last = min(C - 1, (min(row0 + kRows, rows_total) - 1) / gqa);   // last chunk row of the block
  const int n_hist_tiles = (hist + kTile - 1) / kTile;
  const int n_tiles = n_hist_tiles + (i_last + kTile) / kTile;

  // this lane's two query rows (one per column block)
  const int hf = lane >> 5;
  int my_i[kCB];
  bool row_ok[kCB];
  u4 qb[kCB][S::kK];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    const int r = row0 + wave * kRowsPerWave + cb * 32 + (lane & 31);
    row_ok[cb] = r < rows_total;
    my_i[cb] = row_ok[cb] ? r / gqa : 0;
    const int j = row_ok[cb] ? r % gqa : 0;
    const u4* qp = reinterpret_cast<const u4*>(p.q + (((int64_t)b * C + my_i[cb]) * Hq + h * gqa + j) * D);
#pragma unroll
    for (int kk = 0; kk < S::kK; ++kk) qb[cb][kk] = row_ok[cb] ? qp[kk * 2 + hf] : u4(0u);
  }
  // Settle the query loads here, once: the compiler's wait-count pass cannot
  // see the inline-assembly LDS DMAs, so a load still pending at the loop
  // entry would make it wait for vmcnt(0) - every DMA in flight - at the first
  // use of qb on every tile.  Routing qb through an empty asm places that one
  // wait before the loop and leaves no compiler-tracked load behind.
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb)
#pragma unroll
    for (int kk = 0; kk < S::kK; ++kk) asm volatile("" : "+v"(qb[cb][kk]));
  const int wave_i_max = min(C - 1, (min(row0 + wave * kRowsPerWave + kRowsPerWave, rows_total) - 1) / gqa);
  const int wave_i_min = min(C - 1, (row0 + wave * kRowsPerWave) / gqa);

  // DMA of this wave's share (key rows kDmaRows*w .. kDmaRows*(w+1)-1) of tile
  // t into ring slot s
  const uint32_t ring_lds = lds_address(&ring[0][0][0]);
  const int rl = lane / kChunks;   // row within a DMA instruction
  const int pos = lane % kChunks;  // chunk position within the row
  const int rb0 = (wave * kDmaRows) % kPage;   // first row of the share within its page
  auto issue = [&](int t, int s) {
    const uint32_t dst = ring_lds + (uint32_t)s * kTileBytes + (uint32_t)wave * (kDmaRows * kChunks * 16);
    if (t < n_hist_tiles) {
      // past the history: any valid page, masked later
      const int pg = min(t * (kTile / kPage) + wave * kDmaRows / kPage, npages - 1);
      const int64_t id = pt_pages[tbase + pg];
      const u4* kb = p.pool + ((id * 2 + 0) * p.heads_per_group + slot) * (kPage * kChunks);
      const u4* vb = p.pool + ((id * 2 + 1) * p.heads_per_group + slot) * (kPage * kChunks);
#pragma unroll
      for (int j = 0; j < kDmaInst; ++j) {
        const int r = rb0 + j * kRowsPerDma + rl;   // key row within the page (== tile row mod 16)
        lds_dma16(kb + r * kChunks + (pos ^ S::k_swz(r)), dst + j * 1024);
        lds_dma16(vb + r * kChunks + (pos ^ S::v_swz(r)), dst + kTile * kChunks * 16 + j * 1024);
      }
    } else {
      const int c0 = (t - n_hist_tiles) * kTile + wave * kDmaRows;   // first chunk key of the share
      const u4* kb = p.k_new + h * kChunks;
      const u4* vb = p.v_new + h * kChunks;
#pragma unroll
      for (int j = 0; j < kDmaInst; ++j) {
        const int r = j * kRowsPerDma + rl;
        const int c = min(c0 + r, C - 1);   // rows past the chunk repeat its last key (masked later)
        const int rr = rb0 + r;             // tile row mod 16
        const int64_t roff = ((int64_t)b * C + c) * p.num_kv_heads * kChunks;
        lds_dma16(kb + roff + (pos ^ S::k_swz(rr)), dst + j * 1024);
        lds_dma16(vb + roff + (pos ^ S::v_swz(rr)), dst + kTile * kChunks * 16 + j * 1024);
      }
    }
  };

  f32x16 acc[kCB][S::kDB];
  float m[kCB], l[kCB];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
#pragma unroll
    for (int d = 0; d < S::kDB; ++d) acc[cb][d] = f32x16(0.f);
    m[cb] = -INFINITY;
    l[cb] = 0.f;
  }
  const float cs = p.scale_log2;

  // lane-constant parts of the LDS operand addresses
  const int k_row = lane & 31;                                  // A of S^T: key row kb*32 + k_row
  const int tr_key = (lane & 15) >> 2;                          // transposed read: key within a group of 4
  const int tr_dim = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);   // dims within a 32-dim block
  const int tr_chunk = tr_dim >> 3, tr_half = (tr_dim >> 2) & 1;

  // prologue: tiles 0 .. kRing-2 in flight
#pragma unroll
  for (int r = 0; r < kRing - 1; ++r)
    if (r < n_tiles) issue(r, r);

  for (int t = 0; t < n_tiles; ++t) {
    // tile t has landed once at most the DMAs of the tiles after it are pending
    const int after = min(kRing - 2, n_tiles - 1 - t);
    if (after >= 2)
      wait_vmcnt<2 * kDmaPerTile>();
    else if (after == 1)
      wait_vmcnt<kDmaPerTile>();
    else
      wait_vmcnt<0>();
    if (t < n_hist_tiles && t * kTile + wave * kDmaRows + kDmaRows > hist) {
      // this wave's share holds V rows past the retained history: they may
      // hold anything (NaN included) and p = 0 does not cancel NaN, so zero them
      u4* vq = &ring[t % kRing][1][wave * kDmaRows * kChunks];
#pragma unroll
      for (int j = 0; j < kDmaInst; ++j)
        if (t * kTile + wave * kDmaRows + j * kRowsPerDma + rl >= hist) vq[j * 64 + lane] = u4(0u);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
    barrier();   // tile t complete in LDS; every wave is done with tile t-1
    if (t + kRing - 1 < n_tiles) issue(t + kRing - 1, (t + kRing - 1) % kRing);

    const int s = t % kRing;
    const unsigned char* kt = reinterpret_cast<const unsigned char*>(&ring[s][0][0]);
    const unsigned char* vt = reinterpret_cast<const unsigned char*>(&ring[s][1][0]);
    const bool is_chunk = t >= n_hist_tiles;
    const int key0 = is_chunk ? (t - n_hist_tiles) * kTile : t * kTile;   // first key of the tile
    const int key_end = is_chunk ? C : hist;                                 // keys >= this are invalid
    if (is_chunk && key0 > wave_i_max) continue;   // tile entirely in the future of this wave's rows

#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int kbase = key0 + kb * 32;
      if (is_chunk && kbase > wave_i_max) break;
      // S^T for both column blocks; the K operand is read once
      f32x16 sc[kCB];
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb) sc[cb] = f32x16(0.f);
      const int krow = kb * 32 + k_row;
      // all eight K operands of the block, and the V^T operands of its p.v
      // products (they do not depend on p), are requested before the first
      // product, so their LDS latency hides under q.k and the softmax
      u4 ka[S::kK];
#pragma unroll
      for (int kk = 0; kk < S::kK; ++kk)
        ka[kk] = *reinterpret_cast<const u4*>(kt + krow * (2 * D) + (((kk * 2 + hf) ^ S::k_swz(krow)) << 4));
      u4 va[2][S::kDB];
#pragma unroll
      for (int q16 = 0; q16 < 2; ++q16) {
        const int g0 = kb * 32 + q16 * 16 + 4 * hf;    // tile row of the A operand's first key
        const int r0 = g0 + tr_key, r1 = g0 + 8 + tr_key;  // source rows of the two transposed reads
#pragma unroll
        for (int db = 0; db < S::kDB; ++db) {
          const int c = 4 * db + tr_chunk;
          const u2v lo = lds_read_tr16(vt + r0 * (2 * D) + ((c ^ S::v_swz(r0)) << 4) + tr_half * 8);
          const u2v hi = lds_read_tr16(vt + r1 * (2 * D) + ((c ^ S::v_swz(r1)) << 4) + tr_half * 8);
          va[q16][db] = u4{lo.x, lo.y, hi.x, hi.y};
        }
      }
      __builtin_amdgcn_sched_barrier(0);   // keep the reads ahead of the products
#pragma unroll
      for (int kk = 0; kk < S::kK; ++kk)
#pragma unroll
        for (int cb = 0; cb < kCB; ++cb) sc[cb] = mfma(ka[kk], qb[cb][kk], sc[cb]);
      // only the block holding the end of the history and the chunk blocks
      // that reach past the wave's first row need a mask
      const bool masked = is_chunk ? kbase + 31 > wave_i_min : kbase + 32 > hist;
      if (masked) {
#pragma unroll
        for (int cb = 0; cb < kCB; ++cb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            // lane holds keys n(r) = 8*(r/4) + 4*hf + r%4 of its row
            const int key = kbase + 8 * (r >> 2) + 4 * hf + (r & 3);
            const bool ok = key < key_end && (!is_chunk || key <= my_i[cb]);
            sc[cb][r] = ok ? sc[cb][r] : -INFINITY;
          }
      }
      u4 pb[kCB][2];
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb) {
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[cb][r]);
        mx = swap32_max(mx);
        const bool raise = (mx - m[cb]) * cs > kSlack;
        if (__any(raise)) {   // raise the running max (rare after the first block)
          const float m_new = raise ? mx : m[cb];
          const float alpha = fast_exp2((m[cb] - m_new) * cs);   // 0 when m was -inf
          m[cb] = m_new;
          l[cb] *= alpha;
#pragma unroll
          for (int d = 0; d < S::kDB; ++d) acc[cb][d] *= alpha;
        }
        const float mcs = m[cb] * cs;
        uint32_t pw[8];
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const float p0 = fast_exp2(fmaf(sc[cb][r], cs, -mcs));
          const float p1 = fast_exp2(fmaf(sc[cb][r + 1], cs, -mcs));
          l[cb] += p0 + p1;
          pw[r >> 1] = pack_bf16(p0, p1);
        }
        pb[cb][0] = u4{pw[0], pw[1], pw[2], pw[3]};
        pb[cb][1] = u4{pw[4], pw[5], pw[6], pw[7]};
      }
      // O^T += V^T P^T over the two 16-key halves of the block
#pragma unroll
      for (int q16 = 0; q16 < 2; ++q16)
#pragma unroll
        for (int db = 0; db < S::kDB; ++db)
#pragma unroll
          for (int cb = 0; cb < kCB; ++cb) acc[cb][db] = mfma(va[q16][db], pb[cb][q16], acc[cb][db]);
    }
  }
  wait_vmcnt<0>();
  // row sum over both halves of the row, then O = O^T / l
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    const float lt = swap32_sum(l[cb]);
    if (!row_ok[cb]) continue;
    const int r = row0 + wave * kRowsPerWave + cb * 32 + (lane & 31);
    const int i = r / gqa, j = r % gqa;
    const float inv = 1.f / lt;
    uint16_t* orow = p.out + (((int64_t)b * C + i) * Hq + h * gqa + j) * D;
#pragma unroll
    for (int db = 0; db < S::kDB; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int dv = db * 32 + 8 * r4 + 4 * hf;
        const uint32_t w0 = pack_bf16(acc[cb][db][r4 * 4 + 0] * inv, acc[cb][db][r4 * 4 + 1] * inv);
        const uint32_t w1 = pack_bf16(acc[cb][db][r4 * 4 + 2] * inv, acc[cb][db][r4 * 4 + 3] * inv);
        *reinterpret_cast<uint2*>(orow + dv) = make_uint2(w0, w1);
      }
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
  if (g.head_dim != 64 && g.head_dim != 128)
    return tg::fail(TG_ERR_UNSUPPORTED, "prefill supports head_dim 64 or 128 (got %d)", g.head_dim);
  if (g.page_size != kPage) return tg::fail(TG_ERR_UNSUPPORTED, "prefill supports page_size 16 only");
  const int gqa = g.num_q_heads / g.num_kv_heads;
  if (gqa < 1 || gqa > 16) return tg::fail(TG_ERR_UNSUPPORTED, "prefill supports 1..16 query heads per KV head");
  if (a->batch < 1 || a->chunk_len < 1 || a->layer < 0 || a->layer >= g.num_layers)
    return tg::fail(TG_ERR_INVALID_ARG, "batch and chunk_len must be >= 1, layer in range");
  if (!a->q || !a->k_new || !a->v_new || !a->kv_pool || !a->pt_pages || !a->pt_offsets || !a->kv_len ||
      !a->group_of || !a->slot_of || !a->out)
    return tg::fail(TG_ERR_INVALID_ARG, "NULL device pointer");
  if (!tg::aligned16({a->q, a->k_new, a->v_new, a->kv_pool, a->out}))
    return tg::fail(TG_ERR_INVALID_ARG, "device buffers must be 16-byte aligned");
  PrefillParams p;
  p.q = static_cast<const uint16_t*>(a->q);
  p.k_new = static_cast<const u4*>(a->k_new);
  p.v_new = static_cast<const u4*>(a->v_new);
  p.pool = static_cast<const u4*>(a->kv_pool);
  p.pt_pages = a->pt_pages;
  p.pt_offsets = a->pt_offsets;
  p.kv_len = a->kv_len;
  p.group_of = a->group_of;
  p.slot_of = a->slot_of;
  p.out = static_cast<uint16_t*>(a->out);
  p.block_order = a->block_order;
  p.batch = a->batch;
  p.chunk = a->chunk_len;
  p.layer = a->layer;
  p.num_layers = g.num_layers;
  p.num_kv_heads = g.num_kv_heads;
  p.num_groups = g.num_kv_heads / g.heads_per_group;
  p.heads_per_group = g.heads_per_group;
  p.gqa = gqa;
  p.row_tiles = (a->chunk_len * gqa + kRows - 1) / kRows;
  const float scale = a->sm_scale != 0.f ? a->sm_scale : 1.0f / std::sqrt((float)g.head_dim);
  p.scale_log2 = scale * kLog2e;
  const int units = a->batch * g.num_kv_heads;
  if (a->block_order && a->num_blocks < 1) return tg::fail(TG_ERR_INVALID_ARG, "block_order needs num_blocks >= 1");
  const int blocks = a->block_order ? a->num_blocks : 8 * ((units + 7) / 8) * p.row_tiles;
  auto kernel = g.head_dim == 128 ? tg_prefill_kernel<128> : tg_prefill_kernel<64>;
  hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kBlock), 0, static_cast<hipStream_t>(hip_stream), p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "prefill launch failed: %s", hipGetErrorString(e));
  return TG_OK;
}

}  // extern "C"
