// Host-side launchers shared between the C ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/reskv.h"

namespace reskv {

struct DecodePlan {
  int B, Hq, Hkv, G, GP, D, C, Rcap;
  int PR, P;  // residual blocks and all blocks of the split grid per (b, kv head)
  bool whole_head;  // one block per (b, kv head), no split-K records
  size_t acc_off, ml_off, bytes;
};

// Largest dynamic LDS the combine kernel may use for its weights.
size_t decode_max_lds_weights();

DecodePlan make_decode_plan(const reskv_shape_t& s);

hipError_t launch_decode(const reskv_shape_t& s, const reskv_gate_t& g, const DecodePlan& plan,
                         const void* q, void* kc, void* vc, const float* logc,
                         const int32_t* res_len, int32_t* main_len, const void* k_new, const void* v_new,
                         float* out, float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate,
                         void* workspace, hipStream_t stream);

hipError_t launch_append(const reskv_shape_t& s, const void* k_new, const void* v_new, void* kc,
                         void* vc, const int32_t* res_len, int32_t* main_len, hipStream_t stream);

// Construction.
// Sizes of one (b, kv head), fixed on the host from seq_len, budget and r.
struct HeadMeta {
  int s;         // context length
  int r;         // residual entries
  int m;         // main slots of the budget (b - r)
  int P;         // protected recent tokens, min(recent_window, m, s)
  int n_sc;      // scored positions [0, n_sc), s - P
  int k_top;     // top-scored tokens kept, m - P
  int nE;        // evicted tokens, s - m (0 when every token is kept)
  int r_eff;     // Lloyd groups, min(r, nE)
  int main_len;  // min(m, s)
  int all_main;  // 1 when s <= m
};

struct BuildPlan {
  int B, Hq, Hkv, G, D, C, Rcap, S, w, R, T, dtype;
  int NCH;    // scoring key chunks of the longest sequence
  int NBLK;   // 256-token blocks of the largest evicted set
  int max_s, max_main, max_reff;
  size_t off_meta, off_lsep, off_lse, off_raw, off_score, off_elist, off_seeds, off_cent, off_chi,
      off_clo, off_cnorm, off_assign, off_hist, off_cstart, off_ccount, off_order, bytes;
};

bool make_build_plan(const reskv_shape_t& s, const reskv_build_params_t& p, const int32_t* seq_len,
                     const int32_t* budget, const int32_t* res_count, BuildPlan* plan);

hipError_t launch_build(const reskv_shape_t& s, const reskv_build_params_t& p, const BuildPlan& plan,
                        const void* k, const void* v, const int32_t* seq_len, const void* q_obs,
                        const int32_t* budget, const int32_t* res_count, void* kc, void* vc,
                        float* logc, int32_t* main_idx, int32_t* res_len, int32_t* main_len,
                        float* dbg_scores, int32_t* dbg_assign, void* workspace,
                        hipStream_t stream);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace reskv
