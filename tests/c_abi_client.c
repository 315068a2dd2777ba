/* A plain C99 client of libtangram.so: the host calls of the tiny fp32
 * workload (one layer, two requests of 512 tokens, four KV heads with budgets
 * 1, 1/2, 1/4, 1/8, pages of 16, two heads per group) through the C ABI alone,
 * with caller-owned arrays and size queries.  It prints one "key values..."
 * line per result; tests/test_c_client.py compares them with the hand-derived
 * values in tests/golden/config1_hand.json. */
#include <stdio.h>
#include <stdlib.h>

#include "tangram.h"

#define B 2
#define L 1
#define H 4
#define G 2
#define POOL 100

static int check(int32_t rc, const char* what) {
  if (rc != TG_OK) {
    fprintf(stderr, "%s failed: %s (%s)\n", what, tg_status_string(rc), tg_last_error());
    exit(1);
  }
  return 0;
}

static void print_i32(const char* key, const int32_t* v, int n) {
  printf("%s", key);
  for (int i = 0; i < n; ++i) printf(" %d", v[i]);
  printf("\n");
}

#define MAX_ITEMS 128

static void print_plan(const char* key, const tg_geometry* geom, const int32_t* kv_len, const int64_t* offsets,
                       const int32_t* group_of, const int32_t* slot_of, int32_t mode, int32_t want_bins,
                       int32_t split_target) {
  tg_work_item items[MAX_ITEMS];
  int32_t bin_offsets[MAX_ITEMS + 1], unit_splits[B * H], unit_base[B * H], n_items, n_bins, n_partials;
  /* size query first: no item array */
  check(tg_build_plan(geom, B, 0, kv_len, offsets, group_of, slot_of, mode, want_bins, split_target, NULL, NULL, 0,
                      bin_offsets, MAX_ITEMS + 1, unit_splits, unit_base, &n_items, &n_bins, &n_partials),
        "tg_build_plan (size query)");
  if (n_items > MAX_ITEMS || n_bins > MAX_ITEMS) {
    fprintf(stderr, "unexpected plan size %d items, %d bins\n", n_items, n_bins);
    exit(1);
  }
  check(tg_build_plan(geom, B, 0, kv_len, offsets, group_of, slot_of, mode, want_bins, split_target, NULL, items,
                      MAX_ITEMS, bin_offsets, MAX_ITEMS + 1, unit_splits, unit_base, &n_items, &n_bins, &n_partials),
        "tg_build_plan");
  printf("%s_items", key);
  for (int i = 0; i < n_items; ++i)
    printf(" %lld %d %d %d %d %d %d", (long long)items[i].pt_base, items[i].b, items[i].kv_head, items[i].slot,
           items[i].tok_begin, items[i].tok_end, items[i].out_idx);
  printf("\n");
  char k[64];
  snprintf(k, sizeof k, "%s_bin_offsets", key);
  print_i32(k, bin_offsets, n_bins + 1);
  snprintf(k, sizeof k, "%s_unit_splits", key);
  print_i32(k, unit_splits, B * H);
  snprintf(k, sizeof k, "%s_unit_partial_base", key);
  print_i32(k, unit_base, B * H);
  printf("%s_num_partials %d\n", key, n_partials);
  printf("%s_num_bins %d\n", key, n_bins);
}

int main(void) {
  const tg_geometry geom = {L, H, 2 * H, 64, 16, 2};
  const double budget[L * H] = {1.0, 0.5, 0.25, 0.125};
  const int32_t ctx_len[B] = {512, 512};
  int32_t perm[L * H], group_of[L * H], slot_of[L * H];
  int32_t kv_len[B * L * H], group_len[B * L * G], pages[POOL], free_pages[POOL];
  int64_t offsets[B * L * G + 1], pages_needed = 0;
  int32_t S[L * G];

  printf("version %d\n", tg_version());
  check(tg_cluster_heads(&geom, budget, TG_GROUP_CLUSTERED, perm, group_of, slot_of), "tg_cluster_heads");
  print_i32("perm", perm, L * H);
  print_i32("group_of", group_of, L * H);
  print_i32("slot_of", slot_of, L * H);

  for (int i = 0; i < POOL; ++i) free_pages[i] = i;
  /* size query (no page list), then the reservation itself */
  check(tg_reserve(&geom, B, ctx_len, NULL, NULL, budget, group_of, NULL, 0, POOL, kv_len, group_len, offsets, NULL, 0,
                   &pages_needed),
        "tg_reserve (size query)");
  printf("pages_needed_query %lld\n", (long long)pages_needed);
  check(tg_reserve(&geom, B, ctx_len, NULL, NULL, budget, group_of, free_pages, POOL, POOL, kv_len, group_len, offsets,
                   pages, POOL, &pages_needed),
        "tg_reserve");
  printf("pages_needed %lld\n", (long long)pages_needed);
  print_i32("kv_len", kv_len, B * L * H);
  print_i32("group_len", group_len, B * L * G);
  printf("offsets");
  for (int i = 0; i <= B * L * G; ++i) printf(" %lld", (long long)offsets[i]);
  printf("\n");

  check(tg_split_map(&geom, budget, perm, 256, S), "tg_split_map");
  print_i32("split_map_ncta256", S, L * G);
  check(tg_split_map(&geom, budget, perm, 8, S), "tg_split_map");
  print_i32("split_map_ncta8", S, L * G);

  print_plan("plan_aot", &geom, kv_len, offsets, group_of, slot_of, TG_PLAN_AOT, 8, 16);
  print_plan("plan_fill", &geom, kv_len, offsets, group_of, slot_of, TG_PLAN_AOT_FILL, 8, 1);
  print_plan("plan_uniform", &geom, kv_len, offsets, group_of, slot_of, TG_PLAN_UNIFORM, 64, 1);
  print_plan("plan_naive", &geom, kv_len, offsets, group_of, slot_of, TG_PLAN_NAIVE, 64, 1);

  /* an error path: H not divisible by H_p */
  const tg_geometry bad = {L, 3, 6, 64, 16, 2};
  const int32_t rc = tg_cluster_heads(&bad, budget, TG_GROUP_CLUSTERED, perm, group_of, slot_of);
  printf("bad_geometry %d\n", rc);
  return 0;
}
