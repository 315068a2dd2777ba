// Host integer half of libtangram.so: Budget-Aware Clustering, Budget
// Reservation into ragged per-group page tables, Algorithm 1's split map and
// the balanced split-KV partition plan.  Everything here is deterministic
// integer (or exactly specified fp64) work on caller-owned host arrays.
//
// Must be compiled with -ffp-contract=off: the retained length is the IEEE
// fp64 product ceil(r * N) and Algorithm 1's quotients are plain fp64 ops.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <memory>
#include <new>
#include <thread>
#include <queue>
#include <string>
#include <utility>
#include <numeric>
#include <vector>

#include "tg_internal.h"

namespace tg {

static thread_local char g_last_error[512] = "";

int32_t fail(int32_t code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}

int32_t check_geometry(const tg_geometry* g) {
  if (!g) return fail(TG_ERR_INVALID_ARG, "geometry is NULL");
  if (g->num_layers < 1 || g->num_kv_heads < 1 || g->num_q_heads < 1 || g->head_dim < 1 ||
      g->page_size < 1 || g->heads_per_group < 1)
    return fail(TG_ERR_INVALID_ARG, "geometry fields must be >= 1");
  if (g->num_kv_heads % g->heads_per_group != 0)
    return fail(TG_ERR_INVALID_ARG, "num_kv_heads (%d) is not a multiple of heads_per_group (%d)",
                g->num_kv_heads, g->heads_per_group);
  if (g->num_q_heads % g->num_kv_heads != 0)
    return fail(TG_ERR_INVALID_ARG, "num_q_heads (%d) is not a multiple of num_kv_heads (%d)",
                g->num_q_heads, g->num_kv_heads);
  return TG_OK;
}

static bool ratio_ok(double r) { return r > 0.0 && r <= 1.0; }  // false for NaN

}  // namespace tg

// Runs an entry point's body so that no C++ exception reaches a C caller: a
// failed host allocation becomes TG_ERR_NO_MEMORY, anything else
// TG_ERR_INVALID_ARG, with nothing consumed.
template <typename F>
static int32_t guarded(F&& body) {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return tg::fail(TG_ERR_NO_MEMORY, "host memory allocation failed");
  } catch (...) {
    return tg::fail(TG_ERR_INVALID_ARG, "unexpected host error");
  }
}

// Host threads for n independent items: one per 256 Ki items, at most the
// machine's hardware threads and 16 (TG_HOST_THREADS overrides the cap).
static int host_threads(int64_t n) {
  int cap = 16;
  if (const char* e = std::getenv("TG_HOST_THREADS")) cap = std::max(1, std::atoi(e));
  const int hw = std::max(1u, std::thread::hardware_concurrency());
  return (int)std::max<int64_t>(1, std::min<int64_t>({(int64_t)std::min(cap, hw), n >> 18}));
}

// fn(worker, lo, hi) over [0, n) cut into `threads` contiguous chunks; the
// calling thread runs chunk 0, and any chunk whose thread cannot be started.
// No exception leaves: a C caller must never see one.
template <typename F>
static void parallel_chunks(int64_t n, int threads, F fn) {
  if (threads <= 1) {
    fn(0, 0, n);
    return;
  }
  std::vector<std::thread> pool;
  std::vector<int> inline_chunks;
  for (int w = 1; w < threads; ++w) {
    try {
      pool.emplace_back(fn, w, n * w / threads, n * (w + 1) / threads);
    } catch (...) {
      inline_chunks.push_back(w);
    }
  }
  fn(0, 0, n / threads);
  for (int w : inline_chunks) fn(w, n * w / threads, n * (w + 1) / threads);
  for (auto& t : pool) t.join();
}

using tg::ceil_div;
using tg::fail;

// Sequential fill over segments: each segment is a list of units laid end to
// end (in the given order) and cut into its own number of bins whose page
// shares follow the segment's weights (equal when NULL).  Bins are numbered
// across segments in order; a unit cut by a boundary is split, and partial
// indices are numbered over all units in (b, h) order.
//   TG_PLAN_AOT_FILL:  one segment, every unit, n_bins bins (optionally weighted);
//   TG_PLAN_SPLIT_MAP: one segment per head group g (its units in (b, h) order)
//                      with S[layer][g] bins: Algorithm 1's split map as is.
struct FillSegment {
  std::vector<int64_t> units;
  int64_t n_bins;
  const int32_t* weights;
};

static int32_t segmented_fill(int H, int64_t P, int layer, const std::vector<int64_t>& len,
                              const std::vector<int64_t>& base, const int32_t* slot_of,
                              const std::vector<FillSegment>& segs, tg_work_item* items, int32_t item_capacity,
                              int32_t* bin_offsets, int32_t bin_capacity, int32_t* unit_splits,
                              int32_t* unit_partial_base, int32_t* num_items, int32_t* num_bins,
                              int32_t* num_partials) {
  const int64_t n_units = (int64_t)len.size();
  struct Cut {
    std::vector<int64_t> start, cut;
  };
  std::vector<Cut> cuts(segs.size());
  std::vector<int64_t> pieces(n_units, 0);
  int64_t n_items = 0, total_bins = 0;
  for (size_t si = 0; si < segs.size(); ++si) {
    const FillSegment& sg = segs[si];
    Cut& c = cuts[si];
    const int64_t nu = (int64_t)sg.units.size();
    c.start.assign(nu + 1, 0);
    for (int64_t i = 0; i < nu; ++i) c.start[i + 1] = c.start[i] + ceil_div(len[sg.units[i]], P);
    const int64_t total = c.start[nu];
    // bin k covers pages [cut[k], cut[k+1]): cut[k] = floor(total * W_k / W), W_k the
    // weight of the segment's bins before k
    std::vector<int64_t> wsum(sg.n_bins + 1, 0);
    for (int64_t k = 0; k < sg.n_bins; ++k) wsum[k + 1] = wsum[k] + (sg.weights ? sg.weights[k] : 1);
    c.cut.resize(sg.n_bins + 1);
    for (int64_t k = 0; k <= sg.n_bins; ++k) c.cut[k] = (int64_t)((__int128)total * wsum[k] / wsum[sg.n_bins]);
    // count the pieces of every unit (bins walk the units monotonically)
    for (int64_t k = 0, i = 0; k < sg.n_bins; ++k) {
      const int64_t lo = c.cut[k], hi = c.cut[k + 1];
      while (i < nu && c.start[i + 1] <= lo) ++i;
      for (int64_t j = i; j < nu && c.start[j] < hi; ++j)
        if (std::max(lo, c.start[j]) < std::min(hi, c.start[j + 1])) {
          ++pieces[sg.units[j]];
          ++n_items;
        }
    }
    total_bins += sg.n_bins;
  }
  int64_t nparts = 0;
  for (int64_t u = 0; u < n_units; ++u) {
    unit_splits[u] = (int32_t)pieces[u];
    unit_partial_base[u] = pieces[u] > 1 ? (int32_t)nparts : -1;
    if (pieces[u] > 1) nparts += pieces[u];
  }
  if (n_items > INT32_MAX || nparts > INT32_MAX || total_bins > INT32_MAX - 1)
    return fail(TG_ERR_INVALID_ARG, "plan too large");
  *num_items = (int32_t)n_items;
  *num_bins = (int32_t)total_bins;
  *num_partials = (int32_t)nparts;
  if (!items) return TG_OK;  // size query
  if (!bin_offsets) return fail(TG_ERR_INVALID_ARG, "bin_offsets is NULL");
  if (item_capacity < n_items) return fail(TG_ERR_BUFFER_TOO_SMALL, "items holds %d, need %lld", item_capacity, (long long)n_items);
  if (bin_capacity < total_bins + 1)
    return fail(TG_ERR_BUFFER_TOO_SMALL, "bin_offsets holds %d, need %lld", bin_capacity, (long long)(total_bins + 1));
  std::vector<int64_t> seen(n_units, 0);
  int64_t it = 0, bin = 0;
  bin_offsets[0] = 0;
  for (size_t si = 0; si < segs.size(); ++si) {
    const FillSegment& sg = segs[si];
    const Cut& c = cuts[si];
    const int64_t nu = (int64_t)sg.units.size();
    for (int64_t k = 0, i = 0; k < sg.n_bins; ++k) {
      const int64_t lo = c.cut[k], hi = c.cut[k + 1];
      while (i < nu && c.start[i + 1] <= lo) ++i;
      for (int64_t j = i; j < nu && c.start[j] < hi; ++j) {
        const int64_t a = std::max(lo, c.start[j]), z = std::min(hi, c.start[j + 1]);
        if (a >= z) continue;
        const int64_t v = sg.units[j];
        tg_work_item w;
        w.pt_base = base[v];
        w.b = (int32_t)(v / H);
        w.kv_head = (int32_t)(v % H);
        w.slot = slot_of[(int64_t)layer * H + w.kv_head];
        w.tok_begin = (int32_t)((a - c.start[j]) * P);
        w.tok_end = (int32_t)std::min((z - c.start[j]) * P, len[v]);
        w.out_idx = pieces[v] == 1 ? -1 : (int32_t)(unit_partial_base[v] + seen[v]);
        ++seen[v];
        items[it++] = w;
      }
      bin_offsets[++bin] = (int32_t)it;
    }
  }
  return TG_OK;
}

extern "C" {

const char* tg_status_string(int32_t code) {
  switch (code) {
    case TG_OK: return "ok";
    case TG_ERR_INVALID_ARG: return "invalid argument";
    case TG_ERR_OUT_OF_PAGES: return "out of pages";
    case TG_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case TG_ERR_UNSUPPORTED: return "unsupported";
    case TG_ERR_HIP: return "HIP error";
    case TG_ERR_NO_MEMORY: return "out of host memory";
    default: return "unknown status";
  }
}

const char* tg_last_error(void) { return tg::g_last_error; }

int32_t tg_version(void) { return (1 << 16) | 1; }

// Section 4.2.2: sort each layer's heads by ascending budget (stable, so
// equal budgets keep ascending head index) and cut into groups of H_p.
int32_t tg_cluster_heads(const tg_geometry* geom, const double* budget, int32_t grouping,
                         int32_t* perm, int32_t* group_of, int32_t* slot_of) {
  return guarded([&]() -> int32_t {
    if (int32_t rc = tg::check_geometry(geom)) return rc;
    if (!budget || !perm || !group_of || !slot_of) return fail(TG_ERR_INVALID_ARG, "NULL array");
    if (grouping != TG_GROUP_CLUSTERED && grouping != TG_GROUP_ADJACENT)
      return fail(TG_ERR_INVALID_ARG, "unknown grouping %d", grouping);
    const int L = geom->num_layers, H = geom->num_kv_heads, Hp = geom->heads_per_group;
    for (int64_t i = 0; i < (int64_t)L * H; ++i)
      if (!tg::ratio_ok(budget[i])) return fail(TG_ERR_INVALID_ARG, "budget[%lld] outside (0,1]", (long long)i);
    std::vector<int32_t> order(H);
    for (int l = 0; l < L; ++l) {
      const double* bl = budget + (int64_t)l * H;
      for (int h = 0; h < H; ++h) order[h] = h;
      if (grouping == TG_GROUP_CLUSTERED)
        std::stable_sort(order.begin(), order.end(), [bl](int32_t a, int32_t b) { return bl[a] < bl[b]; });
      for (int j = 0; j < H; ++j) {
        const int h = order[j];
        perm[(int64_t)l * H + j] = h;
        group_of[(int64_t)l * H + h] = j / Hp;
        slot_of[(int64_t)l * H + h] = j % Hp;
      }
    }
    return TG_OK;
  });
}

// Eq. 4 + Section 4.1 (Precise Page Allocation) + Section 4.2.1/4.2.3.
int32_t tg_reserve(const tg_geometry* geom, int32_t batch, const int32_t* ctx_len, const int32_t* headroom,
                   const double* ratio, const double* budget, const int32_t* group_of, const int32_t* free_pages,
                   int64_t num_free,
                   int64_t pool_pages, int32_t* kv_len, int32_t* group_len, int64_t* pt_offsets,
                   int32_t* pt_pages, int64_t pt_capacity, int64_t* pages_needed) {
  return guarded([&]() -> int32_t {
    if (int32_t rc = tg::check_geometry(geom)) return rc;
    if (batch < 1) return fail(TG_ERR_INVALID_ARG, "batch must be >= 1");
    if (!ctx_len || !group_of || !kv_len || !group_len || !pt_offsets || !pages_needed)
      return fail(TG_ERR_INVALID_ARG, "NULL array");
    if (!ratio && !budget) return fail(TG_ERR_INVALID_ARG, "ratio and budget are both NULL");
    if (num_free < 0 || pool_pages < 0) return fail(TG_ERR_INVALID_ARG, "negative pool size");
    if (num_free > 0 && !free_pages) return fail(TG_ERR_INVALID_ARG, "free_pages is NULL");
    const int L = geom->num_layers, H = geom->num_kv_heads, G = H / geom->heads_per_group;
    const int64_t P = geom->page_size;
    for (int64_t i = 0; i < (int64_t)L * H; ++i)
      if (group_of[i] < 0 || group_of[i] >= G) return fail(TG_ERR_INVALID_ARG, "group_of[%lld] out of range", (long long)i);
    for (int b = 0; b < batch; ++b) {
      if (ctx_len[b] < 1) return fail(TG_ERR_INVALID_ARG, "ctx_len[%d] < 1", b);
      if (headroom && headroom[b] < 0) return fail(TG_ERR_INVALID_ARG, "headroom[%d] < 0", b);
    }
    // retained lengths first (validating every ratio before anything is written)
    for (int b = 0; b < batch; ++b)
      for (int64_t i = 0; i < (int64_t)L * H; ++i) {
        const double r = ratio ? ratio[(int64_t)b * L * H + i] : budget[i];
        if (!tg::ratio_ok(r)) return fail(TG_ERR_INVALID_ARG, "ratio of request %d entry %lld outside (0,1]", b, (long long)i);
      }
    for (int b = 0; b < batch; ++b) {
      const double n = (double)ctx_len[b];
      for (int64_t i = 0; i < (int64_t)L * H; ++i) {
        const double r = ratio ? ratio[(int64_t)b * L * H + i] : budget[i];
        kv_len[(int64_t)b * L * H + i] = (int32_t)std::ceil(r * n);
      }
    }
    // group lengths and the CSR offsets of every (b, l, g) table
    int64_t k = 0;
    for (int b = 0; b < batch; ++b)
      for (int l = 0; l < L; ++l) {
        int32_t* gl = group_len + ((int64_t)b * L + l) * G;
        for (int g = 0; g < G; ++g) gl[g] = 0;
        const int32_t* kl = kv_len + ((int64_t)b * L + l) * H;
        const int32_t* gof = group_of + (int64_t)l * H;
        for (int h = 0; h < H; ++h) gl[gof[h]] = std::max(gl[gof[h]], kl[h]);
        for (int g = 0; g < G; ++g) {
          pt_offsets[((int64_t)b * L + l) * G + g] = k;
          k += ceil_div((int64_t)gl[g] + (headroom ? headroom[b] : 0), P);
        }
      }
    pt_offsets[(int64_t)batch * L * G] = k;
    *pages_needed = k;
    if (!pt_pages) return TG_OK;  // size query: nothing consumed, free list not examined
    if (k > num_free) return fail(TG_ERR_OUT_OF_PAGES, "reservation needs %lld pages, %lld free", (long long)k, (long long)num_free);
    if (pt_capacity < k) return fail(TG_ERR_BUFFER_TOO_SMALL, "pt_pages holds %lld, need %lld", (long long)pt_capacity, (long long)k);
    // the consumed ids must be distinct pages of the pool.  Each thread marks
    // its chunk of the list in a bitmap of its own (plain stores: no atomics,
    // no cache lines shared between threads); then the pool's id range is cut
    // among the threads and each one ORs the bitmaps' words of its range
    // together, flagging any bit set in two of them.  The bitmaps take
    // threads * pool_pages / 8 bytes, kept within 256 MiB by using fewer
    // threads.  On any failure a sequential pass reports the first offending
    // entry, so the message does not depend on timing.
    const int64_t words = (pool_pages + 63) / 64;
    const int64_t map_cap = std::max<int64_t>(1, (int64_t(256) << 20) / std::max<int64_t>(8, words * 8));
    const int nthreads = (int)std::min<int64_t>(host_threads(k), map_cap);
    std::unique_ptr<uint64_t[]> maps(new uint64_t[(size_t)(nthreads * words)]);
    std::vector<uint8_t> bad((size_t)nthreads, 0);
    parallel_chunks(k, nthreads, [&](int w, int64_t lo, int64_t hi) {
      uint64_t* m = maps.get() + (size_t)w * words;
      std::memset(m, 0, (size_t)words * sizeof(uint64_t));
      for (int64_t i = lo; i < hi; ++i) {
        const int32_t p = free_pages[i];
        if (p < 0 || p >= pool_pages) {
          bad[w] = 1;
          return;
        }
        const uint64_t bit = 1ull << (p & 63);
        if (m[p >> 6] & bit) {
          bad[w] = 1;
          return;
        }
        m[p >> 6] |= bit;
      }
    });
    if (std::find(bad.begin(), bad.end(), 1) == bad.end() && nthreads > 1)
      parallel_chunks(words, nthreads, [&](int w, int64_t lo, int64_t hi) {
        for (int64_t j = lo; j < hi; ++j) {
          uint64_t acc = 0;
          for (int t = 0; t < nthreads; ++t) {
            const uint64_t x = maps[(size_t)t * words + j];
            if (acc & x) {
              bad[w] = 1;
              return;
            }
            acc |= x;
          }
        }
      });
  if (std::find(bad.begin(), bad.end(), 1) != bad.end()) {
    std::vector<uint8_t> once((size_t)pool_pages, 0);
    for (int64_t i = 0; i < k; ++i) {
      const int32_t p = free_pages[i];
      if (p < 0 || p >= pool_pages) return fail(TG_ERR_INVALID_ARG, "free_pages[%lld] = %d outside the pool", (long long)i, p);
      if (once[p]) return fail(TG_ERR_INVALID_ARG, "page id %d appears twice in the free list", p);
      once[p] = 1;
    }
  }
  parallel_chunks(k, nthreads, [&](int, int64_t lo, int64_t hi) {
    std::memcpy(pt_pages + lo, free_pages + lo, (size_t)(hi - lo) * sizeof(int32_t));
  });
  return TG_OK;
  });
}

// Algorithm 1's split map: every group of a layer gets workgroups in
// proportion to its share of the layer's summed budget, at least one,
//   S[l][g] = max(1, round(Phi[l][g] / tau[l])),  tau[l] = Omega[l] / n_cta,
// where Omega[l] sums the layer's budgets (heads in index order) and Phi[l][g]
// the budgets of group g's heads (in the clustering's order), all in fp64.
// round() is half away from zero (floor(x + 0.5) for x > 0), so the counts of a
// layer can add up to slightly more or less than n_cta.  Budgets are validated
// to lie in (0, 1], so Omega > 0 and tau > 0.
int32_t tg_split_map(const tg_geometry* geom, const double* budget, const int32_t* perm, int32_t n_cta, int32_t* S) {
  if (int32_t rc = tg::check_geometry(geom)) return rc;
  if (!budget || !perm || !S) return fail(TG_ERR_INVALID_ARG, "NULL array");
  if (n_cta < 1) return fail(TG_ERR_INVALID_ARG, "n_cta must be >= 1");
  const int L = geom->num_layers, H = geom->num_kv_heads, Hp = geom->heads_per_group, G = H / Hp;
  for (int64_t i = 0; i < (int64_t)L * H; ++i) {
    if (!tg::ratio_ok(budget[i])) return fail(TG_ERR_INVALID_ARG, "budget[%lld] outside (0,1]", (long long)i);
    if (perm[i] < 0 || perm[i] >= H) return fail(TG_ERR_INVALID_ARG, "perm[%lld] out of range", (long long)i);
  }
  std::vector<uint8_t> hit(H);
  for (int l = 0; l < L; ++l) {
    std::fill(hit.begin(), hit.end(), 0);
    for (int j = 0; j < H; ++j) {
      if (hit[perm[(int64_t)l * H + j]]) return fail(TG_ERR_INVALID_ARG, "perm of layer %d is not a permutation", l);
      hit[perm[(int64_t)l * H + j]] = 1;
    }
  }
  // a left-to-right fp64 sum (the order fixes the rounding)
  auto add_up = [](auto first, auto last) { return std::accumulate(first, last, 0.0); };
  std::vector<double> sorted(H);
  for (int l = 0; l < L; ++l) {
    const double* bl = budget + (int64_t)l * H;
    const int32_t* pl = perm + (int64_t)l * H;
    const double tau = add_up(bl, bl + H) / (double)n_cta;
    for (int j = 0; j < H; ++j) sorted[j] = bl[pl[j]];   // budgets in group order
    for (int g = 0; g < G; ++g) {
      const double share = add_up(sorted.begin() + g * Hp, sorted.begin() + (g + 1) * Hp) / tau;
      S[(int64_t)l * G + g] = (int32_t)std::max(1.0, std::floor(share + 0.5));
    }
  }
  return TG_OK;
}

// Balanced split-KV partition of one layer (Algorithm 1's rule on the batch).
static int32_t build_plan_core(const tg_geometry* geom, int32_t batch, int32_t layer, const int32_t* kv_len,
                      const int64_t* pt_offsets, const int32_t* group_of, const int32_t* slot_of, int32_t mode,
                      int32_t n_bins, int32_t split_target, const int32_t* bin_weights, tg_work_item* items,
                      int32_t item_capacity,
                      int32_t* bin_offsets, int32_t bin_capacity, int32_t* unit_splits, int32_t* unit_partial_base,
                      int32_t* num_items, int32_t* num_bins, int32_t* num_partials) {
  if (int32_t rc = tg::check_geometry(geom)) return rc;
  if (!kv_len || !pt_offsets || !group_of || !slot_of || !unit_splits || !unit_partial_base || !num_items ||
      !num_bins || !num_partials)
    return fail(TG_ERR_INVALID_ARG, "NULL array");
  const int L = geom->num_layers, H = geom->num_kv_heads, Hp = geom->heads_per_group, G = H / Hp;
  const int64_t P = geom->page_size;
  if (batch < 1) return fail(TG_ERR_INVALID_ARG, "batch must be >= 1");
  if (layer < 0 || layer >= L) return fail(TG_ERR_INVALID_ARG, "layer %d out of range", layer);
  if (mode != TG_PLAN_AOT && mode != TG_PLAN_NAIVE && mode != TG_PLAN_UNIFORM && mode != TG_PLAN_AOT_FILL &&
      mode != TG_PLAN_SPLIT_MAP)
    return fail(TG_ERR_INVALID_ARG, "unknown plan mode %d", mode);
  if (mode != TG_PLAN_NAIVE && mode != TG_PLAN_SPLIT_MAP && n_bins < 1)
    return fail(TG_ERR_INVALID_ARG, "n_bins must be >= 1");
  if (mode == TG_PLAN_AOT && split_target < 1) return fail(TG_ERR_INVALID_ARG, "split_target must be >= 1");
  if (bin_weights && mode != TG_PLAN_AOT_FILL && mode != TG_PLAN_SPLIT_MAP)
    return fail(TG_ERR_INVALID_ARG, "bin_weights apply to TG_PLAN_AOT_FILL and TG_PLAN_SPLIT_MAP only");
  if (mode == TG_PLAN_SPLIT_MAP && !bin_weights)
    return fail(TG_ERR_INVALID_ARG, "TG_PLAN_SPLIT_MAP needs the layer's split map row in bin_weights");
  if (bin_weights) {
    const int32_t nw = mode == TG_PLAN_SPLIT_MAP ? geom->num_kv_heads / geom->heads_per_group : n_bins;
    for (int32_t k = 0; k < nw; ++k)
      if (bin_weights[k] < 1 || bin_weights[k] > 65535)
        return fail(TG_ERR_INVALID_ARG, "bin_weights[%d] = %d outside [1, 65535]", k, bin_weights[k]);
  }
  const int64_t n_units = (int64_t)batch * H;
  // lengths of this layer, checked against the capacity of their table
  std::vector<int64_t> len(n_units), base(n_units);
  int64_t W = 0;
  for (int b = 0; b < batch; ++b)
    for (int h = 0; h < H; ++h) {
      const int64_t u = (int64_t)b * H + h;
      const int g = group_of[(int64_t)layer * H + h];
      const int s = slot_of[(int64_t)layer * H + h];
      if (g < 0 || g >= G || s < 0 || s >= Hp) return fail(TG_ERR_INVALID_ARG, "group_of/slot_of out of range");
      const int64_t t = ((int64_t)b * L + layer) * G + g;
      const int64_t cap = (pt_offsets[t + 1] - pt_offsets[t]) * P;
      len[u] = kv_len[((int64_t)b * L + layer) * H + h];
      if (len[u] < 1 || len[u] > cap)
        return fail(TG_ERR_INVALID_ARG, "kv_len of request %d head %d (%lld) outside [1, table capacity %lld]", b, h,
                    (long long)len[u], (long long)cap);
      base[u] = pt_offsets[t];
      W += len[u];
    }
  if (mode == TG_PLAN_AOT_FILL || mode == TG_PLAN_SPLIT_MAP) {
    std::vector<FillSegment> segs;
    if (mode == TG_PLAN_AOT_FILL) {
      FillSegment sg{std::vector<int64_t>(n_units), n_bins, bin_weights};
      for (int64_t u = 0; u < n_units; ++u) sg.units[u] = u;
      segs.push_back(std::move(sg));
    } else {
      for (int g = 0; g < G; ++g) {
        FillSegment sg{{}, bin_weights[g], nullptr};
        for (int b = 0; b < batch; ++b)
          for (int h = 0; h < H; ++h)
            if (group_of[(int64_t)layer * H + h] == g) sg.units.push_back((int64_t)b * H + h);
        segs.push_back(std::move(sg));
      }
    }
    return segmented_fill(H, P, layer, len, base, slot_of, segs, items, item_capacity, bin_offsets, bin_capacity,
                          unit_splits, unit_partial_base, num_items, num_bins, num_partials);
  }
  // split counts
  std::vector<int64_t> splits(n_units);
  int64_t total = 0, nparts = 0;
  for (int64_t u = 0; u < n_units; ++u) {
    const int64_t n = ceil_div(len[u], P);
    int64_t s;
    if (mode == TG_PLAN_AOT)
      s = std::max<int64_t>(1, (2 * len[u] * (int64_t)split_target + W) / (2 * W));
    else if (mode == TG_PLAN_NAIVE)
      s = 1;
    else
      s = std::max<int64_t>(1, ceil_div(n_bins, n_units));
    s = std::min(s, n);
    splits[u] = s;
    total += s;
    unit_splits[u] = (int32_t)s;
    unit_partial_base[u] = s > 1 ? (int32_t)nparts : -1;
    if (s > 1) nparts += s;
  }
  const int64_t bins = mode == TG_PLAN_AOT ? n_bins : (mode == TG_PLAN_NAIVE ? n_units : total);
  if (total > INT32_MAX || nparts > INT32_MAX) return fail(TG_ERR_INVALID_ARG, "plan too large");
  *num_items = (int32_t)total;
  *num_bins = (int32_t)bins;
  *num_partials = (int32_t)nparts;
  if (!items) return TG_OK;  // size query
  if (!bin_offsets) return fail(TG_ERR_INVALID_ARG, "bin_offsets is NULL");
  if (item_capacity < total) return fail(TG_ERR_BUFFER_TOO_SMALL, "items holds %d, need %lld", item_capacity, (long long)total);
  if (bin_capacity < bins + 1) return fail(TG_ERR_BUFFER_TOO_SMALL, "bin_offsets holds %d, need %lld", bin_capacity, (long long)(bins + 1));

  // chunks in (b, h, c) order
  std::vector<tg_work_item> chunks;
  chunks.reserve((size_t)total);
  for (int b = 0; b < batch; ++b)
    for (int h = 0; h < H; ++h) {
      const int64_t u = (int64_t)b * H + h, n = ceil_div(len[u], P), s = splits[u];
      for (int64_t c = 0; c < s; ++c) {
        const int64_t p0 = c * n / s, p1 = (c + 1) * n / s;
        tg_work_item it;
        it.pt_base = base[u];
        it.b = b;
        it.kv_head = h;
        it.slot = slot_of[(int64_t)layer * H + h];
        it.tok_begin = (int32_t)(p0 * P);
        it.tok_end = (int32_t)std::min(p1 * P, len[u]);
        it.out_idx = s == 1 ? -1 : (int32_t)(unit_partial_base[u] + c);
        chunks.push_back(it);
      }
    }
  if (mode != TG_PLAN_AOT) {
    // every chunk is its own bin, in (b, h, c) order
    for (int64_t i = 0; i < total; ++i) {
      items[i] = chunks[i];
      bin_offsets[i] = (int32_t)i;
    }
    bin_offsets[total] = (int32_t)total;
    return TG_OK;
  }
  // longest first; ties by (b, h, c), i.e. by position in `chunks`
  std::vector<int32_t> order((size_t)total);
  for (int64_t i = 0; i < total; ++i) order[i] = (int32_t)i;
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return (chunks[a].tok_end - chunks[a].tok_begin) > (chunks[b].tok_end - chunks[b].tok_begin);
  });
  // greedy: least-loaded bin, ties to the lowest bin index
  using Slot = std::pair<int64_t, int32_t>;
  std::priority_queue<Slot, std::vector<Slot>, std::greater<Slot>> heap;
  for (int32_t k = 0; k < n_bins; ++k) heap.push({0, k});
  std::vector<int32_t> bin_of((size_t)total), count((size_t)n_bins, 0);
  for (int64_t i = 0; i < total; ++i) {
    Slot s = heap.top();
    heap.pop();
    const tg_work_item& c = chunks[order[i]];
    bin_of[i] = s.second;
    count[s.second] += 1;
    heap.push({s.first + (c.tok_end - c.tok_begin), s.second});
  }
  bin_offsets[0] = 0;
  for (int32_t k = 0; k < n_bins; ++k) bin_offsets[k + 1] = bin_offsets[k] + count[k];
  std::vector<int32_t> fill(bin_offsets, bin_offsets + n_bins);
  for (int64_t i = 0; i < total; ++i) items[fill[bin_of[i]]++] = chunks[order[i]];
  return TG_OK;
}

int32_t tg_build_plan(const tg_geometry* geom, int32_t batch, int32_t layer, const int32_t* kv_len,
                      const int64_t* pt_offsets, const int32_t* group_of, const int32_t* slot_of, int32_t mode,
                      int32_t n_bins, int32_t split_target, const int32_t* bin_weights, tg_work_item* items,
                      int32_t item_capacity, int32_t* bin_offsets, int32_t bin_capacity, int32_t* unit_splits,
                      int32_t* unit_partial_base, int32_t* num_items, int32_t* num_bins, int32_t* num_partials) {
  return guarded([&]() -> int32_t {
    if ((mode & ~0x1ff) != 0) return fail(TG_ERR_INVALID_ARG, "unknown plan mode %d", mode);
    const bool open_end = (mode & TG_PLAN_OPEN_END) != 0;
    const int32_t rc = build_plan_core(geom, batch, layer, kv_len, pt_offsets, group_of, slot_of,
                                       mode & ~TG_PLAN_OPEN_END, n_bins, split_target, bin_weights, items,
                                       item_capacity, bin_offsets, bin_capacity, unit_splits, unit_partial_base,
                                       num_items, num_bins, num_partials);
    if (rc != TG_OK || !open_end || !items) return rc;
    // the chunk that ends each unit runs to the live length, bounded by its table
    const int64_t L = geom->num_layers, H = geom->num_kv_heads, G = H / geom->heads_per_group;
    for (int32_t i = 0; i < *num_items; ++i) {
      tg_work_item& it = items[i];
      const int64_t lh = (int64_t)layer * H + it.kv_head;
      if (it.tok_end != kv_len[((int64_t)it.b * L + layer) * H + it.kv_head]) continue;
      const int64_t t = ((int64_t)it.b * L + layer) * G + group_of[lh];
      it.tok_end = (int32_t)(-(pt_offsets[t + 1] - pt_offsets[t]) * geom->page_size);
    }
    return TG_OK;
  });
}

// Ahead-of-time workgroup schedule of tg_prefill: LPT placement of the
// (request, KV head) units on the XCDs, longest blocks first on each XCD.
int32_t tg_prefill_schedule(const tg_geometry* geom, int32_t batch, int32_t chunk_len, int32_t layer,
                            const int32_t* kv_len, int32_t n_xcd, int32_t* order, int32_t capacity,
                            int32_t* num_blocks) {
  return guarded([&]() -> int32_t {
    if (int32_t rc = tg::check_geometry(geom)) return rc;
    if (!kv_len || !num_blocks) return fail(TG_ERR_INVALID_ARG, "NULL array");
    if (batch < 1 || chunk_len < 1) return fail(TG_ERR_INVALID_ARG, "batch and chunk_len must be >= 1");
    if (layer < 0 || layer >= geom->num_layers) return fail(TG_ERR_INVALID_ARG, "layer %d out of range", layer);
    if (n_xcd < 1 || n_xcd > 64) return fail(TG_ERR_INVALID_ARG, "n_xcd must be in 1..64");
    const int64_t L = geom->num_layers, H = geom->num_kv_heads, gqa = geom->num_q_heads / geom->num_kv_heads;
    const int64_t C = chunk_len, rows = C * gqa;
    const int64_t row_tiles = tg::ceil_div(rows, TG_PREFILL_ROWS);
    const int64_t n_units = (int64_t)batch * H;
    if (n_units * row_tiles > INT32_MAX / 2) return fail(TG_ERR_INVALID_ARG, "too many prefill blocks");
    // cost of every block and unit
    std::vector<int64_t> chunk_tiles(row_tiles), unit_cost(n_units);
    for (int64_t rt = 0; rt < row_tiles; ++rt) {
      const int64_t i_last = std::min(C - 1, (std::min((rt + 1) * TG_PREFILL_ROWS, rows) - 1) / gqa);
      chunk_tiles[rt] = i_last / TG_PREFILL_TILE + 1;
    }
    std::vector<int64_t> hist_tiles(n_units);
    for (int64_t u = 0; u < n_units; ++u) {
      const int64_t b = u / H, h = u % H;
      const int64_t len = kv_len[(b * L + layer) * H + h];
      if (len < 0) return fail(TG_ERR_INVALID_ARG, "negative kv_len at request %lld head %lld", (long long)b,
                               (long long)h);
      hist_tiles[u] = tg::ceil_div(len, TG_PREFILL_TILE);
      unit_cost[u] = 0;
      for (int64_t rt = 0; rt < row_tiles; ++rt) unit_cost[u] += hist_tiles[u] + chunk_tiles[rt];
    }
    // units to XCDs, longest first, each to the least-loaded XCD (ties: lowest index)
    std::vector<int64_t> units(n_units);
    for (int64_t u = 0; u < n_units; ++u) units[u] = u;
    std::stable_sort(units.begin(), units.end(),
                     [&](int64_t a, int64_t b) { return unit_cost[a] > unit_cost[b]; });
    std::vector<int64_t> load(n_xcd, 0);
    std::vector<std::vector<std::pair<int64_t, int64_t>>> blocks(n_xcd);   // (u, rt)
    for (int64_t u : units) {
      int x = 0;
      for (int k = 1; k < n_xcd; ++k)
        if (load[k] < load[x]) x = k;
      load[x] += unit_cost[u];
      for (int64_t rt = 0; rt < row_tiles; ++rt) blocks[x].emplace_back(u, rt);
    }
    size_t longest = 0;
    for (auto& v : blocks) {
      std::stable_sort(v.begin(), v.end(), [&](const std::pair<int64_t, int64_t>& a, const std::pair<int64_t, int64_t>& b) {
        const int64_t ca = hist_tiles[a.first] + chunk_tiles[a.second];
        const int64_t cb = hist_tiles[b.first] + chunk_tiles[b.second];
        if (ca != cb) return ca > cb;
        return a < b;
      });
      longest = std::max(longest, v.size());
    }
    const int64_t total = (int64_t)n_xcd * (int64_t)longest;
    *num_blocks = (int32_t)total;
    if (!order) return TG_OK;   // size query
    if (capacity < total) return fail(TG_ERR_BUFFER_TOO_SMALL, "order holds %d, need %lld", capacity, (long long)total);
    for (int64_t k = 0; k < total; ++k) {
      const auto& v = blocks[k % n_xcd];
      const size_t j = (size_t)(k / n_xcd);
      order[k] = j < v.size() ? (int32_t)(v[j].first * row_tiles + v[j].second) : -1;
    }
    return TG_OK;
  });
}

}  // extern "C"

// Compression fused into chunked prefill (Section 4.1): after x context tokens
// a head holds ceil(r*x) entries (Eq. 4 on the prefix, one fp64 multiply and
// ceil), never more than its reservation; a chunk keeps the difference.
extern "C" int32_t tg_compress_plan(const tg_geometry* geom, int32_t batch, int32_t layer, int32_t chunk_len,
                                    const int32_t* chunk_start, const int32_t* chunk_tokens, const double* ratio,
                                    const double* budget, const int32_t* kv_len, const int64_t* pt_offsets,
                                    const int32_t* group_of, const int32_t* slot_of, int32_t rows_per_item,
                                    tg_compress_item* items, int32_t item_capacity, int32_t* keep_count,
                                    int32_t* write_begin, int32_t* num_items) {
  return guarded([&]() -> int32_t {
    if (int32_t rc = tg::check_geometry(geom)) return rc;
    if (batch < 1) return fail(TG_ERR_INVALID_ARG, "batch must be >= 1");
    const int L = geom->num_layers, H = geom->num_kv_heads, Hp = geom->heads_per_group, G = H / Hp;
    const int64_t P = geom->page_size;
    if (layer < 0 || layer >= L) return fail(TG_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, L);
    if (chunk_len < 1 || chunk_len > TG_COMPRESS_MAX_CHUNK)
      return fail(TG_ERR_INVALID_ARG, "chunk_len %d outside [1, %d]", chunk_len, (int)TG_COMPRESS_MAX_CHUNK);
    if (rows_per_item < 1 || rows_per_item > TG_COMPRESS_MAX_ROWS)
      return fail(TG_ERR_INVALID_ARG, "rows_per_item %d outside [1, %d]", rows_per_item, (int)TG_COMPRESS_MAX_ROWS);
    if (!chunk_start || !chunk_tokens || !kv_len || !pt_offsets || !group_of || !slot_of || !keep_count ||
        !write_begin || !num_items)
      return fail(TG_ERR_INVALID_ARG, "NULL array");
    if (!ratio && !budget) return fail(TG_ERR_INVALID_ARG, "ratio and budget are both NULL");
    if (item_capacity < 0) return fail(TG_ERR_INVALID_ARG, "negative item_capacity");
    for (int h = 0; h < H; ++h) {
      const int64_t i = (int64_t)layer * H + h;
      if (group_of[i] < 0 || group_of[i] >= G || slot_of[i] < 0 || slot_of[i] >= Hp)
        return fail(TG_ERR_INVALID_ARG, "group_of / slot_of of head %d out of range", h);
    }
    // validate everything before writing anything
    for (int b = 0; b < batch; ++b) {
      if (chunk_start[b] < 0) return fail(TG_ERR_INVALID_ARG, "chunk_start[%d] < 0", b);
      if (chunk_tokens[b] < 0 || chunk_tokens[b] > chunk_len)
        return fail(TG_ERR_INVALID_ARG, "chunk_tokens[%d] = %d outside [0, %d]", b, chunk_tokens[b], chunk_len);
      if ((int64_t)chunk_start[b] + chunk_tokens[b] > INT32_MAX)
        return fail(TG_ERR_INVALID_ARG, "chunk_start + chunk_tokens of request %d overflows int32", b);
      for (int h = 0; h < H; ++h) {
        const int64_t i = ((int64_t)b * L + layer) * H + h;
        const double r = ratio ? ratio[i] : budget[(int64_t)layer * H + h];
        if (!tg::ratio_ok(r)) return fail(TG_ERR_INVALID_ARG, "ratio of request %d head %d outside (0,1]", b, h);
        if (kv_len[i] < 0) return fail(TG_ERR_INVALID_ARG, "kv_len of request %d head %d < 0", b, h);
        const int64_t t = ((int64_t)b * L + layer) * G + group_of[(int64_t)layer * H + h];
        if ((pt_offsets[t + 1] - pt_offsets[t]) * P < kv_len[i])
          return fail(TG_ERR_INVALID_ARG, "page table of request %d head %d holds fewer than kv_len entries", b, h);
      }
    }
    int64_t n_items = 0;
    for (int b = 0; b < batch; ++b) {
      const double c0 = (double)chunk_start[b], c1 = (double)chunk_start[b] + (double)chunk_tokens[b];
      for (int h = 0; h < H; ++h) {
        const int64_t i = ((int64_t)b * L + layer) * H + h;
        const double r = ratio ? ratio[i] : budget[(int64_t)layer * H + h];
        const int64_t cap = kv_len[i];
        const int64_t cursor = std::min((int64_t)std::ceil(r * c0), cap);
        const int64_t end = std::min((int64_t)std::ceil(r * c1), cap);
        keep_count[(int64_t)b * H + h] = (int32_t)(end - cursor);
        write_begin[(int64_t)b * H + h] = (int32_t)cursor;
        n_items += ceil_div(end - cursor, rows_per_item);
      }
    }
    if (n_items > INT32_MAX) return fail(TG_ERR_INVALID_ARG, "too many work items");
    *num_items = (int32_t)n_items;
    if (!items) return TG_OK;
    if (item_capacity < n_items)
      return fail(TG_ERR_BUFFER_TOO_SMALL, "items holds %d, need %lld", item_capacity, (long long)n_items);
    int64_t k = 0;
    for (int b = 0; b < batch; ++b)
      for (int h = 0; h < H; ++h) {
        const int32_t cnt = keep_count[(int64_t)b * H + h];
        const int64_t lh = (int64_t)layer * H + h;
        const int64_t base = pt_offsets[((int64_t)b * L + layer) * G + group_of[lh]];
        for (int32_t r0 = 0; r0 < cnt; r0 += rows_per_item) {
          tg_compress_item& it = items[k++];
          it.pt_base = base;
          it.b = b;
          it.kv_head = h;
          it.slot = slot_of[lh];
          it.n_valid = chunk_tokens[b];
          it.cursor = write_begin[(int64_t)b * H + h];
          it.count = cnt;
          it.rank_begin = r0;
          it.rank_end = std::min(cnt, r0 + rows_per_item);
        }
      }
    return TG_OK;
  });
}

// KV slots allocated by each paging scheme for the same retained lengths
// (Section 4.2.1: a table spans one group; PagedAttention spans all L x H heads).
extern "C" int32_t tg_memory_footprint(const tg_geometry* geom, int32_t batch, const int32_t* ctx_len,
                                       const double* ratio, const double* budget, const int32_t* group_of,
                                       tg_footprint* out) {
  return guarded([&]() -> int32_t {
    if (int32_t rc = tg::check_geometry(geom)) return rc;
    if (batch < 1) return fail(TG_ERR_INVALID_ARG, "batch must be >= 1");
    if (!ctx_len || !group_of || !out) return fail(TG_ERR_INVALID_ARG, "NULL array");
    if (!ratio && !budget) return fail(TG_ERR_INVALID_ARG, "ratio and budget are both NULL");
    const int L = geom->num_layers, H = geom->num_kv_heads, Hp = geom->heads_per_group, G = H / Hp;
    const int64_t P = geom->page_size;
    for (int64_t i = 0; i < (int64_t)L * H; ++i)
      if (group_of[i] < 0 || group_of[i] >= G) return fail(TG_ERR_INVALID_ARG, "group_of[%lld] out of range", (long long)i);
    for (int b = 0; b < batch; ++b) {
      if (ctx_len[b] < 1) return fail(TG_ERR_INVALID_ARG, "ctx_len[%d] < 1", b);
      for (int64_t i = 0; i < (int64_t)L * H; ++i) {
        const double r = ratio ? ratio[(int64_t)b * L * H + i] : budget[i];
        if (!tg::ratio_ok(r)) return fail(TG_ERR_INVALID_ARG, "ratio of request %d entry %lld outside (0,1]", b, (long long)i);
      }
    }
    tg_footprint f = {0, 0, 0, 0, 0, (int64_t)batch * L * G};
    std::vector<int64_t> gl(G);
    for (int b = 0; b < batch; ++b) {
      const double n = (double)ctx_len[b];
      f.full_slots += ceil_div(ctx_len[b], P) * P * L * H;
      int64_t longest = 0;
      for (int l = 0; l < L; ++l) {
        std::fill(gl.begin(), gl.end(), 0);
        for (int h = 0; h < H; ++h) {
          const int64_t i = (int64_t)l * H + h;
          const double r = ratio ? ratio[(int64_t)b * L * H + i] : budget[i];
          const int64_t len = (int64_t)std::ceil(r * n);
          f.retained_slots += len;
          longest = std::max(longest, len);
          gl[group_of[i]] = std::max(gl[group_of[i]], len);
        }
        for (int g = 0; g < G; ++g) {
          const int64_t pages = ceil_div(gl[g], P);
          f.ragged_pages += pages;
          f.ragged_slots += pages * P * Hp;
        }
      }
      f.monolithic_slots += ceil_div(longest, P) * P * L * H;
    }
    *out = f;
    return TG_OK;
  });
}

// Order-preserving 32-bit key of an fp32 score: larger number, larger key;
// -0 and +0 share a key; NaN gets 0, below -inf.
static inline uint32_t score_key(float f) {
  uint32_t u;
  std::memcpy(&u, &f, sizeof(u));
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Implicit per-head retention ratios of one sample (Eq. 3's layer-wide top-k).
extern "C" int32_t tg_implicit_ratios(int32_t num_layers, int32_t num_heads, int32_t n_tokens, const float* scores,
                                      double rho, double* ratios, int32_t* counts) {
  return guarded([&]() -> int32_t {
    if (num_layers < 1 || num_heads < 1 || n_tokens < 1) return fail(TG_ERR_INVALID_ARG, "L, H and N must be >= 1");
    if ((int64_t)num_heads * n_tokens >= INT32_MAX) return fail(TG_ERR_INVALID_ARG, "H * N too large");
    if (!(rho > 0.0 && rho <= 1.0)) return fail(TG_ERR_INVALID_ARG, "rho outside (0, 1]");
    if (!scores || !ratios) return fail(TG_ERR_INVALID_ARG, "NULL array");
    const int64_t HN = (int64_t)num_heads * n_tokens;
    const int64_t k = (int64_t)std::ceil(rho * (double)HN);
    // composite key: score key, then the lower flattened index first (a total order)
    std::vector<uint64_t> key((size_t)HN), sorted;
    for (int l = 0; l < num_layers; ++l) {
      const float* s = scores + (int64_t)l * HN;
      for (int64_t i = 0; i < HN; ++i)
        key[i] = ((uint64_t)score_key(s[i]) << 32) | (uint64_t)(0xffffffffu - (uint32_t)i);
      sorted = key;
      std::nth_element(sorted.begin(), sorted.begin() + (k - 1), sorted.end(), std::greater<uint64_t>());
      const uint64_t kth = sorted[k - 1];
      for (int h = 0; h < num_heads; ++h) {
        int64_t c = 0;
        for (int64_t t = 0; t < n_tokens; ++t) c += key[(int64_t)h * n_tokens + t] >= kth;
        ratios[(int64_t)l * num_heads + h] = (double)c / (double)n_tokens;
        if (counts) counts[(int64_t)l * num_heads + h] = (int32_t)c;
      }
    }
    return TG_OK;
  });
}

// B = min(1, mu + alpha * sigma) over the samples, at least floor.
extern "C" int32_t tg_calibrate_budget(int32_t samples, int32_t num_layers, int32_t num_heads, const double* ratios,
                                       double alpha, double floor, double* budget) {
  if (samples < 1 || num_layers < 1 || num_heads < 1) return fail(TG_ERR_INVALID_ARG, "S, L and H must be >= 1");
  if (!(alpha >= 0.0) || !(floor > 0.0 && floor <= 1.0)) return fail(TG_ERR_INVALID_ARG, "alpha < 0 or floor outside (0, 1]");
  if (!ratios || !budget) return fail(TG_ERR_INVALID_ARG, "NULL array");
  const int64_t LH = (int64_t)num_layers * num_heads;
  for (int64_t i = 0; i < LH * samples; ++i)
    if (!(ratios[i] >= 0.0 && ratios[i] <= 1.0)) return fail(TG_ERR_INVALID_ARG, "ratio %lld outside [0, 1]", (long long)i);
  for (int64_t i = 0; i < LH; ++i) {
    double acc = 0.0;
    for (int s = 0; s < samples; ++s) acc += ratios[(int64_t)s * LH + i];
    const double mu = acc / samples;
    double var = 0.0;
    for (int s = 0; s < samples; ++s) {
      const double dev = ratios[(int64_t)s * LH + i] - mu;
      var += dev * dev;
    }
    const double sigma = std::sqrt(var / samples);
    const double b = mu + alpha * sigma;
    budget[i] = std::max(floor, std::min(1.0, b));
  }
  return TG_OK;
}

// Finished requests give their pages back; the survivors' tables are compacted.
extern "C" int32_t tg_release_requests(const tg_geometry* geom, int32_t batch, const int64_t* pt_offsets,
                                       const int32_t* pt_pages, const uint8_t* finished, int32_t* freed,
                                       int64_t freed_capacity, int64_t* new_offsets, int32_t* new_pages,
                                       int64_t pages_capacity, int64_t* num_freed, int64_t* num_kept,
                                       int32_t* num_survivors) {
  if (int32_t rc = tg::check_geometry(geom)) return rc;
  if (batch < 1) return fail(TG_ERR_INVALID_ARG, "batch must be >= 1");
  if (!pt_offsets || !finished || !num_freed || !num_kept || !num_survivors) return fail(TG_ERR_INVALID_ARG, "NULL array");
  const int64_t per = (int64_t)geom->num_layers * (geom->num_kv_heads / geom->heads_per_group);
  if (pt_offsets[0] != 0) return fail(TG_ERR_INVALID_ARG, "pt_offsets must start at 0");
  for (int64_t t = 0; t < batch * per; ++t)
    if (pt_offsets[t + 1] < pt_offsets[t]) return fail(TG_ERR_INVALID_ARG, "pt_offsets decreases at %lld", (long long)t);
  int64_t nf = 0, nk = 0;
  int32_t ns = 0;
  for (int b = 0; b < batch; ++b) {
    const int64_t n = pt_offsets[(b + 1) * per] - pt_offsets[b * per];
    if (finished[b]) {
      nf += n;
    } else {
      nk += n;
      ++ns;
    }
  }
  *num_freed = nf;
  *num_kept = nk;
  *num_survivors = ns;
  if (!freed && !new_pages) return TG_OK;  // size query
  if (!freed || !new_pages || !new_offsets || !pt_pages) return fail(TG_ERR_INVALID_ARG, "NULL output array");
  if (freed_capacity < nf || pages_capacity < nk) return fail(TG_ERR_BUFFER_TOO_SMALL, "output arrays too small");
  int64_t f = 0, k = 0, t_out = 0;
  for (int b = 0; b < batch; ++b) {
    const int64_t lo = pt_offsets[b * per], hi = pt_offsets[(b + 1) * per];
    if (finished[b]) {
      std::memcpy(freed + f, pt_pages + lo, (size_t)(hi - lo) * sizeof(int32_t));
      f += hi - lo;
    } else {
      for (int64_t t = 0; t < per; ++t) new_offsets[t_out++] = pt_offsets[b * per + t] - lo + k;
      std::memcpy(new_pages + k, pt_pages + lo, (size_t)(hi - lo) * sizeof(int32_t));
      k += hi - lo;
    }
  }
  new_offsets[t_out] = k;
  return TG_OK;
}

// The tables of batch b appended after those of batch a.
extern "C" int32_t tg_concat_tables(const tg_geometry* geom, int32_t batch_a, const int64_t* offsets_a,
                                    const int32_t* pages_a, int32_t batch_b, const int64_t* offsets_b,
                                    const int32_t* pages_b, int64_t* offsets, int32_t* pages) {
  if (int32_t rc = tg::check_geometry(geom)) return rc;
  if (batch_a < 0 || batch_b < 0) return fail(TG_ERR_INVALID_ARG, "negative batch");
  if (!offsets_a || !offsets_b || !offsets) return fail(TG_ERR_INVALID_ARG, "NULL array");
  const int64_t per = (int64_t)geom->num_layers * (geom->num_kv_heads / geom->heads_per_group);
  const int64_t na = offsets_a[(int64_t)batch_a * per], nb = offsets_b[(int64_t)batch_b * per];
  if (offsets_a[0] != 0 || offsets_b[0] != 0 || na < 0 || nb < 0) return fail(TG_ERR_INVALID_ARG, "bad offsets");
  if ((na > 0 && !pages_a) || (nb > 0 && !pages_b) || (na + nb > 0 && !pages)) return fail(TG_ERR_INVALID_ARG, "NULL pages");
  for (int64_t t = 0; t < (int64_t)batch_a * per; ++t) offsets[t] = offsets_a[t];
  for (int64_t t = 0; t <= (int64_t)batch_b * per; ++t) offsets[(int64_t)batch_a * per + t] = offsets_b[t] + na;
  if (na) std::memcpy(pages, pages_a, (size_t)na * sizeof(int32_t));
  if (nb) std::memcpy(pages + na, pages_b, (size_t)nb * sizeof(int32_t));
  return TG_OK;
}
