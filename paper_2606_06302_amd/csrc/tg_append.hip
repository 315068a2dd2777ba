// Decode-token append: one decode step's new token of one layer, written after
// every KV head's current entries in its group's reserved pages (Tangram's
// ragged layout, Section 4.2), with the head's live length advanced by one.
//
// A group of row_u4 lanes (16-byte vectors per K or V row: 8, 16 or 32) owns
// one (request, KV head) unit; 256 / row_u4 units per workgroup.  The unit
// reads its live length n, checks it against the capacity of its page table,
// copies its K and V rows into entry n and publishes n + 1 from its first lane
// after the rows are stored.
#include <hip/hip_runtime.h>

#include "tg_internal.h"

namespace {

constexpr int kThreads = 256;

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

struct AppendParams {
  const u4* k_tok;
  const u4* v_tok;
  u4* pool;
  const int32_t* pt_pages;
  const int64_t* pt_offsets;
  const int32_t* group_of;
  const int32_t* slot_of;
  int32_t* live_len;
  int32_t* full;
  int32_t batch, L, H, G, Hp, P, layer;
  int32_t row_u4;
};

__global__ __launch_bounds__(kThreads) void tg_append_kernel(AppendParams p) {
  const int lpr = p.row_u4;
  const int units_per_wg = kThreads / lpr;
  const int64_t unit = (int64_t)blockIdx.x * units_per_wg + threadIdx.x / lpr;
  const int sub = threadIdx.x % lpr;
  if (unit >= (int64_t)p.batch * p.H) return;
  const int b = (int)(unit / p.H), h = (int)(unit % p.H);
  const int64_t lh = (int64_t)p.layer * p.H + h;
  int32_t* live = p.live_len + ((int64_t)b * p.L + p.layer) * p.H + h;
  const int n = *live;
  const int64_t t = ((int64_t)b * p.L + p.layer) * p.G + p.group_of[lh];
  const int64_t base = p.pt_offsets[t];
  const int64_t cap = (p.pt_offsets[t + 1] - base) * p.P;
  if (n < 0 || n >= cap) {
    if (p.full && sub == 0) *p.full = 1;
    return;
  }
  const int64_t page = p.pt_pages[base + n / p.P];
  const int64_t dst = ((page * 2 * p.Hp + p.slot_of[lh]) * p.P + n % p.P) * lpr + sub;
  const int64_t src = unit * lpr + sub;
  p.pool[dst] = p.k_tok[src];
  p.pool[dst + (int64_t)p.Hp * p.P * lpr] = p.v_tok[src];
  // every lane of the unit has read n (same wave, same load); the rows are
  // ordered before the length by the kernel boundary for later launches
  if (sub == 0) *live = n + 1;
}

}  // namespace

extern "C" int32_t tg_append(const tg_append_args* a, void* hip_stream) {
  if (!a) return tg::fail(TG_ERR_INVALID_ARG, "args is NULL");
  const tg_geometry& g = a->geom;
  if (int32_t rc = tg::check_geometry(&g)) return rc;
  if (a->dtype != TG_F32 && a->dtype != TG_BF16) return tg::fail(TG_ERR_UNSUPPORTED, "dtype must be f32 or bf16");
  if (g.head_dim != 64 && g.head_dim != 128)
    return tg::fail(TG_ERR_UNSUPPORTED, "append supports head_dim 64 or 128 (got %d)", g.head_dim);
  if (a->batch < 1) return tg::fail(TG_ERR_INVALID_ARG, "batch must be >= 1");
  if (a->layer < 0 || a->layer >= g.num_layers) return tg::fail(TG_ERR_INVALID_ARG, "layer %d out of range", a->layer);
  if (!a->k_tok || !a->v_tok || !a->kv_pool || !a->pt_pages || !a->pt_offsets || !a->group_of || !a->slot_of ||
      !a->live_len)
    return tg::fail(TG_ERR_INVALID_ARG, "NULL device pointer");
  if (!tg::aligned16({a->k_tok, a->v_tok, a->kv_pool}))
    return tg::fail(TG_ERR_INVALID_ARG, "device buffers must be 16-byte aligned");
  AppendParams p;
  p.k_tok = static_cast<const u4*>(a->k_tok);
  p.v_tok = static_cast<const u4*>(a->v_tok);
  p.pool = static_cast<u4*>(a->kv_pool);
  p.pt_pages = a->pt_pages;
  p.pt_offsets = a->pt_offsets;
  p.group_of = a->group_of;
  p.slot_of = a->slot_of;
  p.live_len = a->live_len;
  p.full = a->full;
  p.batch = a->batch;
  p.L = g.num_layers;
  p.H = g.num_kv_heads;
  p.Hp = g.heads_per_group;
  p.G = g.num_kv_heads / g.heads_per_group;
  p.P = g.page_size;
  p.layer = a->layer;
  p.row_u4 = g.head_dim * (a->dtype == TG_F32 ? 4 : 2) / 16;
  const int64_t units = (int64_t)a->batch * g.num_kv_heads;
  const int64_t per_wg = kThreads / p.row_u4;
  const int64_t blocks = (units + per_wg - 1) / per_wg;
  if (blocks > INT32_MAX) return tg::fail(TG_ERR_INVALID_ARG, "batch too large");
  hipLaunchKernelGGL(tg_append_kernel, dim3((unsigned)blocks), dim3(kThreads), 0,
                     static_cast<hipStream_t>(hip_stream), p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tg::fail(TG_ERR_HIP, "append launch failed: %s", hipGetErrorString(e));
  return TG_OK;
}
