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
  size_t acc_off, ml_off, bytes;
};

// Largest dynamic LDS the combine kernel may use for its weights.
size_t decode_max_lds_weights();

DecodePlan make_decode_plan(const reskv_shape_t& s);

hipError_t launch_decode(const reskv_shape_t& s, const reskv_gate_t& g, const DecodePlan& plan,
                         const void* q, const void* kc, const void* vc, const float* logc,
                         const int32_t* res_len, const int32_t* main_len, float* out,
                         float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate,
                         void* workspace, hipStream_t stream);

hipError_t launch_append(const reskv_shape_t& s, const void* k_new, const void* v_new, void* kc,
                         void* vc, const int32_t* res_len, int32_t* main_len, hipStream_t stream);

// Construction.
struct BuildPlan {
  int B, Hq, Hkv, G, D, C, Rcap, S, w, T, dtype;
  // per-(b, kv head) host-side sizes
  int max_s, max_scored, max_E, max_r;
  size_t bytes;
  size_t off_lse, off_raw, off_score, off_meta, off_elist, off_seeds, off_cent, off_assign,
      off_cnt, off_perm, off_sum, off_hist, off_misc;
  int n_lse_parts;  // key chunks of the LSE pass
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
