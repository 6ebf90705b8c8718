/* Host-side exercise of the ResKV C ABI for the sanitizer build: workspace
 * sizes for valid arguments and the argument checks of every entry point.
 * Every call here returns before anything is launched, so no GPU is needed. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "reskv.h"

static int fails = 0;
#define EXPECT(cond)                                        \
  do {                                                      \
    if (!(cond)) {                                          \
      fprintf(stderr, "line %d: %s\n", __LINE__, #cond);    \
      ++fails;                                              \
    }                                                       \
  } while (0)

int main(void) {
  reskv_shape_t sh = {2, 8, 2, 128, RESKV_BF16, 640, 64};
  reskv_build_params_t bp = {300, 16, 16, 4, 0, 0};
  int32_t seq[2] = {300, 200}, bud[2] = {64, 48}, res[4] = {13, 0, 47, 1};
  double grid[5] = {0.0, 0.05, 0.10, 0.15, 0.20};
  reskv_proxy_params_t px = {grid, 5, 4, 0.01f};
  reskv_gate_t gate = {NULL, 0.25f, 12.0f, 0.0f, 1.0f};
  char dummy[64];
  void* p = dummy;

  /* valid sizes */
  EXPECT(reskv_decode_workspace_size(&sh) > 0);
  EXPECT(reskv_build_workspace_size(&sh, &bp, seq, bud, res) > 0);
  EXPECT(reskv_build_adakv_workspace_size(&sh, &bp, 0.2, 0, seq, bud, res) > 0);
  EXPECT(reskv_build_adakv_workspace_size(&sh, &bp, 0.2, 64, seq, bud, res) > 0);
  EXPECT(reskv_build_proxy_workspace_size(&sh, &bp, &px, seq, bud) > 0);

  /* invalid shapes and parameters: sizes are 0, calls return errors */
  reskv_shape_t bad = sh;
  bad.head_dim = 96;
  EXPECT(reskv_decode_workspace_size(&bad) == 0);
  EXPECT(reskv_decode_attn(&bad, &gate, p, p, p, p, p, p, NULL, NULL, p, NULL, NULL, NULL, p, 64, NULL) ==
         RESKV_ERR_UNSUPPORTED);
  bad = sh;
  bad.num_q_heads = 7;
  EXPECT(reskv_build_cache(&bad, &bp, p, p, seq, p, bud, res, p, p, p, p, p, p, NULL, NULL, NULL, p, 64, NULL) ==
         RESKV_ERR_INVALID_ARG);
  EXPECT(strlen(reskv_last_error()) > 0);
  reskv_gate_t bg = gate;
  bg.g_min = 2.0f;
  EXPECT(reskv_decode_attn(&sh, &bg, p, p, p, p, p, p, NULL, NULL, p, NULL, NULL, NULL, p, 1 << 30, NULL) ==
         RESKV_ERR_INVALID_ARG);
  EXPECT(reskv_decode_attn(&sh, &gate, p, p, p, p, p, p, NULL, NULL, p, NULL, NULL, NULL, p, 8, NULL) ==
         RESKV_ERR_WORKSPACE);
  int32_t bres[4] = {64, 0, 0, 0}; /* r >= budget */
  EXPECT(reskv_build_workspace_size(&sh, &bp, seq, bud, bres) == 0);
  EXPECT(reskv_build_cache(&sh, &bp, p, p, seq, p, bud, bres, p, p, p, p, p, p, NULL, NULL, NULL, p, 1 << 30, NULL) ==
         RESKV_ERR_INVALID_ARG);
  EXPECT(reskv_build_cache_adakv(&sh, &bp, 1.5, 0, p, p, seq, p, bud, res, p, p, p, p, p, p, NULL, NULL, NULL, p,
                                 1 << 30, NULL) == RESKV_ERR_INVALID_ARG);
  EXPECT(reskv_build_adakv_workspace_size(&sh, &bp, NAN, 0, seq, bud, res) == 0);
  /* the decode reserve must leave every budget inside the slot capacity */
  EXPECT(reskv_build_adakv_workspace_size(&sh, &bp, 0.2, 577, seq, bud, res) == 0);
  EXPECT(reskv_build_adakv_workspace_size(&sh, &bp, 0.2, -1, seq, bud, res) == 0);
  EXPECT(reskv_build_cache_adakv(&sh, &bp, 0.2, 577, p, p, seq, p, bud, res, p, p, p, p, p, p, NULL, NULL, NULL, p,
                                 1 << 30, NULL) == RESKV_ERR_INVALID_ARG);
  double nogrid[2] = {0.05, 0.1}; /* no zero fraction */
  reskv_proxy_params_t bpx = {nogrid, 2, 4, 0.01f};
  EXPECT(reskv_build_proxy_workspace_size(&sh, &bp, &bpx, seq, bud) == 0);
  EXPECT(reskv_build_cache_proxy(&sh, &bp, &bpx, &gate, p, p, seq, p, bud, p, p, p, p, p, p, NULL, p, 1 << 30,
                                 NULL) == RESKV_ERR_INVALID_ARG);
  EXPECT(reskv_merge_branches(&sh, 5, p, p, p, p, p, p, NULL) == RESKV_ERR_INVALID_ARG);
  EXPECT(reskv_append_kv(&sh, NULL, p, p, p, p, p, NULL) == RESKV_ERR_INVALID_ARG);
  EXPECT(reskv_decode_branches(&sh, &gate, p, p, p, p, p, p, p, p, p, p, p, p, 8, NULL) == RESKV_ERR_WORKSPACE);
  EXPECT(reskv_decode_attn(NULL, &gate, p, p, p, p, p, p, NULL, NULL, p, NULL, NULL, NULL, p, 64, NULL) ==
         RESKV_ERR_INVALID_ARG);
  for (int st = 0; st <= 5; ++st) EXPECT(reskv_status_string((reskv_status_t)st) != NULL);

  if (fails) return 1;
  puts("abi host check: ok");
  return 0;
}
