// Host-side launchers shared between the C ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <vector>

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

// Size of the file-scope device scratch of the allocation-free decode entry
// point, and the current device's address of it (looked up once per device).
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
hipError_t static_scratch(void** ptr);

DecodePlan make_decode_plan(const reskv_shape_t& s);

// Ragged schedule: balanced ranges of 64-slot units over the whole batch.
struct RaggedPlan {
  int BH, GP, blocks;  // blocks launched (enough for any lengths the capacity allows)
  int min_units;       // units per block at least (a head spans at most 64 blocks)
  size_t plan_off, rec_off, bytes;
};
bool make_ragged_plan(const reskv_shape_t& s, RaggedPlan* plan);
hipError_t launch_decode_ragged(const reskv_shape_t& s, const reskv_gate_t& g, const RaggedPlan& pl,
                                const void* q, void* kc, void* vc, const float* logc, const int32_t* res_len,
                                int32_t* main_len, const void* k_new, const void* v_new, float* out,
                                float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate, void* workspace,
                                hipStream_t stream);

hipError_t launch_decode(const reskv_shape_t& s, const reskv_gate_t& g, const DecodePlan& plan,
                         const void* q, void* kc, void* vc, const float* logc,
                         const int32_t* res_len, int32_t* main_len, const void* k_new, const void* v_new,
                         float* out, float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate,
                         void* workspace, hipStream_t stream);

// The two branches of one decode step under their own softmax (split path).
hipError_t launch_decode_branches(const reskv_shape_t& s, const reskv_gate_t& g, const DecodePlan& pl,
                                  const void* q, const void* kc, const void* vc, const float* logc,
                                  const int32_t* res_len, const int32_t* main_len, float* out_main,
                                  float* lse_main, float* out_res, float* lse_res, float* gate_out,
                                  void* workspace, hipStream_t stream);

hipError_t launch_merge_branches(const reskv_shape_t& s, int mode, const float* out_main, const float* lse_main,
                                 const float* out_res, const float* lse_res, const float* gate, float* out,
                                 hipStream_t stream);

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
  int B, Hq, Hkv, G, D, C, Rcap, S, w, T, dtype;
  int wr;     // leading window rows per query head that score
  int pool_half;  // score pooling taps on each side
  int R;      // scoring rows per kv head, G * wr
  int LG;     // 256-key groups per lse block
  int NCH;    // lse key chunks (256 * LG keys) of the longest sequence
  int NSC;    // score-pass key chunks of the longest sequence
  int NBLK;   // 256-token blocks of the largest evicted set
  int NSEL;   // selection blocks (8192 scores each) of the longest sequence
  int max_s, max_main, max_reff, max_E;
  size_t off_meta, off_lsep, off_lse, off_raw, off_score, off_elist, off_seeds, off_cent, off_chi,
      off_clo, off_cnorm, off_assign, off_hist, off_cstart, off_ccount, off_order, off_selh, off_selc, bytes;
};

// Device buffers one construction writes.
struct BuildOut {
  void* kc;
  void* vc;
  float* logc;
  int32_t* main_idx;
  int32_t* res_len;
  int32_t* main_len;
};

bool make_build_plan(const reskv_shape_t& s, const reskv_build_params_t& p, const int32_t* seq_len,
                     const int32_t* budget, const int32_t* res_count, BuildPlan* plan);

// Plan pieces: sizes from the shape, maxima over one or more sets of head
// sizes (several candidate counts fold into one plan), workspace layout.
void init_build_plan(const reskv_shape_t& s, const reskv_build_params_t& p, BuildPlan* plan);
void head_meta(const BuildPlan& pl, const int32_t* seq_len, const int32_t* budget, const int32_t* res_count,
               int recent, std::vector<HeadMeta>& out);
bool fold_build_plan(const std::vector<HeadMeta>& hm, BuildPlan* plan);
bool layout_build_plan(BuildPlan* plan);

// Writes the head sizes of res_count[B*Hkv] to meta[B*Hkv] on the stream.
hipError_t upload_meta(const BuildPlan& pl, const int32_t* seq_len, const int32_t* budget,
                       const int32_t* res_count, int recent, HeadMeta* meta, hipStream_t stream);
// Raw window scores into the workspace, for the scored positions of `meta`.
hipError_t launch_build_scores(const BuildPlan& pl, const void* k, const void* q_obs, const HeadMeta* meta,
                               void* workspace, hipStream_t stream);
// Pooling, selection, gather and Lloyd rounds from the workspace's raw
// scores, for the counts of `meta`, writing `out`.
hipError_t launch_build_candidate(const BuildPlan& pl, const void* k, const void* v, const HeadMeta* meta,
                                  const BuildOut& out, float* dbg_scores, int32_t* dbg_assign, float* dbg_centers,
                                  void* workspace, hipStream_t stream);

// AdaKV cross-head allocation (App. B.2.2 compared methods): at most this
// many KV heads per sequence share their budgets.
constexpr int kAdaMaxHeads = 32;

// Plan whose grids cover every allocation the cross-head step can make: a
// head may hold up to min(s, C' - r) main slots (C' = C - decode_reserve) and
// as few as floor(safeguard * k_top) + |P|.
bool make_build_plan_adakv(const reskv_shape_t& s, const reskv_build_params_t& p, double safeguard,
                           int decode_reserve, const int32_t* seq_len, const int32_t* budget,
                           const int32_t* res_count, BuildPlan* plan);

hipError_t launch_build_adakv(const reskv_shape_t& s, const reskv_build_params_t& p, double safeguard,
                              int decode_reserve, const BuildPlan& plan, const void* k, const void* v,
                              const int32_t* seq_len, const void* q_obs, const int32_t* budget,
                              const int32_t* res_count, void* kc, void* vc, float* logc, int32_t* main_idx,
                              int32_t* res_len, int32_t* main_len, float* dbg_scores, int32_t* dbg_assign,
                              float* dbg_centers, void* workspace, hipStream_t stream);

hipError_t launch_build(const reskv_shape_t& s, const reskv_build_params_t& p, const BuildPlan& plan,
                        const void* k, const void* v, const int32_t* seq_len, const void* q_obs,
                        const int32_t* budget, const int32_t* res_count, void* kc, void* vc,
                        float* logc, int32_t* main_idx, int32_t* res_len, int32_t* main_len,
                        float* dbg_scores, int32_t* dbg_assign, float* dbg_centers, void* workspace,
                        hipStream_t stream);

// Validation proxy (Sec. 5.5.1; App. D, Algorithm 1).
constexpr int kProxyMaxGrid = 8;

struct ProxyPlan {
  BuildPlan build;          // scratch of one candidate build, sized for every candidate
  int NG;                   // candidates
  int val;                  // validation rows per query head
  int GV;                   // validation queries per kv head, G * val
  int NQC, GC;              // query chunks of at most 16 queries, queries per chunk
  std::vector<int32_t> counts;  // [NG][B*Hkv] candidate counts
  std::vector<int32_t> r_max;   // [B*Hkv] largest candidate count (its scored positions cover all)
  DecodePlan dec_full, dec_cand;
  size_t off_meta;          // [NG + 1][B*Hkv] HeadMeta (candidates, then scoring)
  size_t off_kc, off_vc;    // [NG*B][Hkv][C][d]
  size_t off_logc;          // [NG*B][Hkv][Rcap]
  size_t off_midx;          // [NG*B][Hkv][C]
  size_t off_rlen, off_mlen;    // [NG*B*Hkv]
  size_t off_rlen0, off_mlen0, off_logc0;  // [B*Hkv] lengths of the uncompressed prefix
  size_t off_q;             // [NQC][NG*B][Hkv*GC][d] validation queries
  size_t off_out_full;      // [NQC][B][Hkv*GC][d] fp32
  size_t off_out_cand;      // [NQC][NG*B][Hkv*GC][d] fp32
  size_t off_dec;           // decode split-K scratch
  size_t off_loss;          // [NG][B*Hkv] fp32
  size_t off_choice;        // [B*Hkv] int32
  size_t bytes;
};

bool make_proxy_plan(const reskv_shape_t& s, const reskv_build_params_t& p, const reskv_proxy_params_t& x,
                     const int32_t* seq_len, const int32_t* budget, ProxyPlan* plan);

hipError_t launch_build_proxy(const reskv_shape_t& s, const reskv_build_params_t& p,
                              const reskv_proxy_params_t& x, const reskv_gate_t& g, const ProxyPlan& pl,
                              const void* k, const void* v, const int32_t* seq_len, const void* q_obs,
                              const int32_t* budget, void* kc, void* vc, float* logc, int32_t* main_idx,
                              int32_t* res_len, int32_t* main_len, float* val_loss, void* workspace,
                              hipStream_t stream);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace reskv
