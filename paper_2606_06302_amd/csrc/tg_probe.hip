// Streaming-read ceiling of the decode access pattern (diagnostic).
//
// Entry i names one (page, slot): its K slab and its V slab, P * d elements
// each, at the page layout of the ragged cache.  The entries are cut into
// n_workers contiguous ranges, one per wave; a wave reads its slabs with
// 16-byte vector loads, two (K, V) slab pairs in flight, folds every word
// into an XOR and stores one checksum word.  Few registers per wave, so many
// waves per SIMD keep loads in flight.  No arithmetic beyond the XOR and no
// LDS: the time is the time to stream the bytes.  The loads are non-temporal,
// the cache policy of the decode kernel's page reads.
#include <hip/hip_runtime.h>

#include "tg_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / 64;
constexpr int kUnroll = 2;            // slab pairs in flight per wave

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

struct ProbeParams {
  const u4* pool;
  const int32_t* page_ids;
  const int32_t* slots;
  uint32_t* out;
  int64_t n;
  int32_t n_workers;
  int32_t slab_u4;       // 16-byte vectors per slab
  int32_t hp;            // slots per page
};

// PL = 16-byte vectors per lane per slab (slab of 64 * PL * 16 bytes)
template <int PL>
__global__ __launch_bounds__(kThreads) void tg_read_probe_kernel(ProbeParams p) {
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (w >= p.n_workers) return;
  const int64_t lo = p.n * w / p.n_workers, hi = p.n * (w + 1) / p.n_workers;
  u4 x = u4(0u);
  for (int64_t e = lo; e < hi; e += kUnroll) {
    u4 v[kUnroll][2][PL];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (e + u < hi) {
        const int64_t page = p.page_ids[e + u];
        const int64_t slot = p.slots[e + u];
        const u4* k = p.pool + ((page * 2 + 0) * p.hp + slot) * p.slab_u4;
        const u4* vv = p.pool + ((page * 2 + 1) * p.hp + slot) * p.slab_u4;
#pragma unroll
        for (int j = 0; j < PL; ++j) {
          v[u][0][j] = __builtin_nontemporal_load(k + j * 64 + lane);
          v[u][1][j] = __builtin_nontemporal_load(vv + j * 64 + lane);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (e + u < hi)
#pragma unroll
        for (int j = 0; j < PL; ++j) x ^= v[u][0][j] ^ v[u][1][j];
  }
  uint32_t r = x.x ^ x.y ^ x.z ^ x.w;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) r ^= __shfl_xor(r, o, 64);
  if (lane == 0) p.out[w] = r;
}

}  // namespace

extern "C" int32_t tg_read_probe(const tg_geometry* geom, int32_t dtype, const void* kv_pool, const int32_t* page_ids,
                                 const int32_t* slots, int64_t n, int32_t n_workers, uint32_t* out,
                                 void* hip_stream) {
  if (int32_t rc = tg::check_geometry(geom)) return rc;
  if (dtype != TG_F32 && dtype != TG_BF16) return tg::fail(TG_ERR_UNSUPPORTED, "dtype must be f32 or bf16");
  const int64_t slab_bytes = (int64_t)geom->page_size * geom->head_dim * (dtype == TG_F32 ? 4 : 2);
  // the kernel is instantiated for slabs of 2, 4 and 8 KiB (2, 4 or 8 16-byte loads per lane)
  if (slab_bytes != 2048 && slab_bytes != 4096 && slab_bytes != 8192)
    return tg::fail(TG_ERR_UNSUPPORTED, "slab of %lld bytes: need 2, 4 or 8 KiB", (long long)slab_bytes);
  if (n < 0 || n_workers < 1) return tg::fail(TG_ERR_INVALID_ARG, "n < 0 or n_workers < 1");
  if (n > 0 && (!kv_pool || !page_ids || !slots)) return tg::fail(TG_ERR_INVALID_ARG, "NULL device pointer");
  if (!tg::aligned16({kv_pool})) return tg::fail(TG_ERR_INVALID_ARG, "device buffers must be 16-byte aligned");
  if (!out) return tg::fail(TG_ERR_INVALID_ARG, "out is NULL");
  ProbeParams p;
  p.pool = static_cast<const u4*>(kv_pool);
  p.page_ids = page_ids;
  p.slots = slots;
  p.out = out;
  p.n = n;
  p.n_workers = n_workers;
  p.slab_u4 = (int32_t)(slab_bytes / 16);
  p.hp = geom->heads_per_group;
  const int blocks = (n_workers + kWavesPerBlock - 1) / kWavesPerBlock;
  const int pl = p.slab_u4 / 64;
  void (*fn)(ProbeParams) = nullptr;
  switch (pl) {
    case 2: fn = tg_read_probe_kernel<2>; break;
    case 4: fn = tg_read_probe_kernel<4>; break;
    case 8: fn = tg_read_probe_kernel<8>; break;
    default: return tg::fail(TG_ERR_UNSUPPORTED, "slab of %lld bytes", (long long)slab_bytes);
  }
  hipLaunchKernelGGL(fn, dim3(blocks), dim3(kThreads), 0, static_cast<hipStream_t>(hip_stream), p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "probe launch failed: %s", hipGetErrorString(e));
  return TG_OK;
}
