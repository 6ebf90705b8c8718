// Construction-time validation proxy (Sec. 5.5.1, validation-loss and margin
// equations; App. D, Algorithm 1).
//
// Per layer, in launch order:
//   scoring        the fit rows score once, for the scored positions of the
//                  largest candidate count (every smaller count scores a
//                  prefix of them; raw scores do not depend on the count)
//   candidates     for each grid count: pooling, selection, gather and Lloyd
//                  rounds into that candidate's own cache in the workspace
//   gather_q       the G * val validation queries of every kv head, in
//                  chunks of at most 16 heads, as decode queries (repeated
//                  once per candidate: candidate c of sequence b is decode
//                  batch row c * B + b)
//   decode         per chunk: the uncompressed prefix [0, s) as a cache with
//                  no residual entries gives o_S; the candidates' caches, one
//                  decode launch for all of them, give o_r
//   loss           mean over the validation queries of ||o_r - o_S||^2
//   choose         least loss among counts > 0 (ties to the smaller count),
//                  kept only under the relative margin, else count 0
//   copy           the chosen candidate's cache into the outputs
#include <math.h>

#include "common.h"
#include "internal.h"

namespace reskv {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxChunkQueries = 16;  // decode handles groups of at most 16 query heads

// Validation query jj = h * val + i of kv head kvh is window row fit + i of
// query head kvh * G + h. Chunk ch holds queries ch*GC .. ch*GC + GC - 1; the
// padding past GV repeats the last query (its outputs are not scored).
struct GatherArgs {
  const void* q_obs;  // [B, Hq, w, d]
  void* qv;           // [NQC][NG*B][Hkv*GC][d]
  int B, Hq, Hkv, G, w, fit, val, GV, GC, NQC, NG;
};

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void proxy_gather_q(GatherArgs a) {
  constexpr int kPieces = D * (int)sizeof(T) / 16;
  const size_t rows = (size_t)a.NQC * a.NG * a.B * a.Hkv * a.GC;
  for (size_t x = blockIdx.x * (size_t)kThreads + threadIdx.x; x < rows * kPieces;
       x += (size_t)gridDim.x * kThreads) {
    const int pc = (int)(x % kPieces);
    size_t row = x / kPieces;
    const int j = (int)(row % a.GC);
    row /= a.GC;
    const int kvh = (int)(row % a.Hkv);
    row /= a.Hkv;
    const int b = (int)(row % a.B);  // row = ch * NG * B + c * B + b
    const int ch = (int)(row / ((size_t)a.NG * a.B));
    int jj = ch * a.GC + j;
    if (jj >= a.GV) jj = a.GV - 1;
    const int h = jj / a.val, i = jj % a.val;
    const T* src = static_cast<const T*>(a.q_obs) + (((size_t)b * a.Hq + kvh * a.G + h) * a.w + a.fit + i) * D;
    T* dst = static_cast<T*>(a.qv) + (x / kPieces) * D;
    reinterpret_cast<uint4*>(dst)[pc] = reinterpret_cast<const uint4*>(src)[pc];
  }
}

// Lengths of the uncompressed prefix read as a cache: no residual entries,
// s main slots.
__global__ __launch_bounds__(kThreads) void proxy_full_lengths(const HeadMeta* meta, int32_t* rlen, int32_t* mlen,
                                                               float* logc, int BH) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= BH) return;
  rlen[i] = 0;
  mlen[i] = meta[i].s;
  logc[i] = -__builtin_huge_valf();
}

// One block per (candidate c, b, kv head): fp64 sum of the squared output
// differences over the chunk elements in a fixed order, divided by GV.
__global__ __launch_bounds__(kThreads) void proxy_loss(const float* out_full, const float* out_cand, float* loss,
                                                       int B, int Hkv, int GC, int GV, int NQC, int NG, int D) {
  const int bh = blockIdx.x, c = blockIdx.y;
  const int b = bh / Hkv, kvh = bh % Hkv;
  const int per_chunk = GC * D;
  double acc = 0.0;
  for (int e = threadIdx.x; e < NQC * per_chunk; e += kThreads) {
    const int ch = e / per_chunk, j = (e / D) % GC, dd = e % D;
    if (ch * GC + j >= GV) continue;
    const size_t ifull = ((((size_t)ch * B + b) * Hkv + kvh) * GC + j) * D + dd;
    const size_t icand = ((((size_t)ch * NG * B + (size_t)c * B + b) * Hkv + kvh) * GC + j) * D + dd;
    const double df = (double)out_cand[icand] - (double)out_full[ifull];
    acc += df * df;
  }
  __shared__ double s_red[kThreads / 64];
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) acc += __shfl_xor(acc, m, 64);
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int w = 0; w < kThreads / 64; ++w) t += s_red[w];
    loss[(size_t)c * B * Hkv + bh] = (float)(t / GV);
  }
}

// One thread per (b, kv head): the margin rule over the candidates' fp32
// losses (grid order; the first count-0 candidate is the reference).
__global__ __launch_bounds__(kThreads) void proxy_choose(const HeadMeta* cmeta, const float* loss, float delta,
                                                         int NG, int BH, int32_t* choice, int32_t* res_len,
                                                         int32_t* main_len, float* val_loss) {
  const int bh = blockIdx.x * kThreads + threadIdx.x;
  if (bh >= BH) return;
  int i0 = -1, best = -1;
  for (int c = 0; c < NG; ++c) {
    const int r = cmeta[(size_t)c * BH + bh].r;
    const float l = loss[(size_t)c * BH + bh];
    if (val_loss) val_loss[(size_t)bh * NG + c] = l;
    if (r == 0) {
      if (i0 < 0) i0 = c;
      continue;
    }
    if (best < 0) { best = c; continue; }
    const float lb = loss[(size_t)best * BH + bh];
    const int rb = cmeta[(size_t)best * BH + bh].r;
    if (l < lb || (l == lb && r < rb)) best = c;
  }
  int pick = i0 < 0 ? 0 : i0;  // the host guarantees a count-0 candidate
  if (best >= 0 && i0 >= 0) {
    const float thr = (1.0f - delta) * loss[(size_t)i0 * BH + bh];
    if (loss[(size_t)best * BH + bh] < thr) pick = best;
  }
  const HeadMeta m = cmeta[(size_t)pick * BH + bh];
  choice[bh] = pick;
  res_len[bh] = m.r;
  main_len[bh] = m.main_len;
}

// Copies the chosen candidate's slots [0, r + main_len), log-counts and main
// indices into the outputs.
struct CopyArgs {
  const HeadMeta* cmeta;
  const int32_t* choice;
  const void* kc_c;
  const void* vc_c;
  const float* logc_c;
  const int32_t* midx_c;
  void* kc;
  void* vc;
  float* logc;
  int32_t* main_idx;
  int B, Hkv, C, Rcap;
};

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void proxy_copy(CopyArgs a) {
  const int kvh = blockIdx.y, b = blockIdx.z;
  const int BH = a.B * a.Hkv, bh = b * a.Hkv + kvh;
  const int c = a.choice[bh];
  const HeadMeta m = a.cmeta[(size_t)c * BH + bh];
  const size_t src_bh = (size_t)c * BH + bh;  // candidate c of sequence b is decode row c * B + b
  constexpr int kPieces = D * (int)sizeof(T) / 16;
  const int rows = m.r + m.main_len;
  const uint4* ks = reinterpret_cast<const uint4*>(static_cast<const T*>(a.kc_c) + src_bh * a.C * D);
  const uint4* vs = reinterpret_cast<const uint4*>(static_cast<const T*>(a.vc_c) + src_bh * a.C * D);
  uint4* kd = reinterpret_cast<uint4*>(static_cast<T*>(a.kc) + (size_t)bh * a.C * D);
  uint4* vd = reinterpret_cast<uint4*>(static_cast<T*>(a.vc) + (size_t)bh * a.C * D);
  for (int x = blockIdx.x * kThreads + threadIdx.x; x < rows * kPieces; x += gridDim.x * kThreads) {
    kd[x] = ks[x];
    vd[x] = vs[x];
  }
  for (int j = blockIdx.x * kThreads + threadIdx.x; j < a.Rcap; j += gridDim.x * kThreads)
    a.logc[(size_t)bh * a.Rcap + j] = a.logc_c[src_bh * a.Rcap + j];
  for (int i = blockIdx.x * kThreads + threadIdx.x; i < m.main_len; i += gridDim.x * kThreads)
    a.main_idx[(size_t)bh * a.C + i] = a.midx_c[src_bh * a.C + i];
}

reskv_shape_t full_shape(const ProxyPlan& pl) {
  const BuildPlan& b = pl.build;
  return reskv_shape_t{b.B, b.Hkv * pl.GC, b.Hkv, b.D, b.dtype, b.S, 1};
}

reskv_shape_t cand_shape(const ProxyPlan& pl) {
  const BuildPlan& b = pl.build;
  return reskv_shape_t{pl.NG * b.B, b.Hkv * pl.GC, b.Hkv, b.D, b.dtype, b.C, b.Rcap};
}

template <typename T, int D>
hipError_t launch_tail_typed(const ProxyPlan& pl, const GatherArgs& ga, const CopyArgs& ca, hipStream_t st,
                             int stage) {
  const BuildPlan& b = pl.build;
  if (stage == 0) {
    const size_t pieces = (size_t)pl.NQC * pl.NG * b.B * b.Hkv * pl.GC * (D * sizeof(T) / 16);
    size_t blocks = (pieces + kThreads - 1) / kThreads;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL((proxy_gather_q<T, D>), dim3((unsigned)blocks), dim3(kThreads), 0, st, ga);
  } else {
    const int rows = b.max_main + b.Rcap;
    int blocks = (rows * (D * (int)sizeof(T) / 16) + kThreads - 1) / kThreads;
    if (blocks > 64) blocks = 64;
    hipLaunchKernelGGL((proxy_copy<T, D>), dim3(blocks < 1 ? 1 : blocks, b.Hkv, b.B), dim3(kThreads), 0, st, ca);
  }
  return hipGetLastError();
}

hipError_t launch_tail(const ProxyPlan& pl, const GatherArgs& ga, const CopyArgs& ca, hipStream_t st, int stage) {
  const bool bf = pl.build.dtype == RESKV_BF16;
  if (pl.build.D == 128)
    return bf ? launch_tail_typed<uint16_t, 128>(pl, ga, ca, st, stage) : launch_tail_typed<float, 128>(pl, ga, ca, st, stage);
  if (pl.build.D == 64)
    return bf ? launch_tail_typed<uint16_t, 64>(pl, ga, ca, st, stage) : launch_tail_typed<float, 64>(pl, ga, ca, st, stage);
  return hipErrorInvalidValue;
}

}  // namespace

bool make_proxy_plan(const reskv_shape_t& s, const reskv_build_params_t& p, const reskv_proxy_params_t& x,
                     const int32_t* seq_len, const int32_t* budget, ProxyPlan* plan) {
  ProxyPlan& pl = *plan;
  pl = ProxyPlan{};
  reskv_build_params_t pf = p;
  pf.fit_rows = p.obs_window - x.val_rows;
  init_build_plan(s, pf, &pl.build);
  BuildPlan& bp = pl.build;
  const int BH = bp.B * bp.Hkv;
  pl.NG = x.n_grid;
  pl.val = x.val_rows;
  pl.GV = bp.G * x.val_rows;
  pl.NQC = (pl.GV + kMaxChunkQueries - 1) / kMaxChunkQueries;
  pl.GC = (pl.GV + pl.NQC - 1) / pl.NQC;
  // candidate counts r = floor(f * b + 1/2), the same for the kv heads of a sequence
  pl.counts.assign((size_t)pl.NG * BH, 0);
  pl.r_max.assign(BH, 0);
  for (int c = 0; c < pl.NG; ++c)
    for (int bh = 0; bh < BH; ++bh) {
      const int r = (int)floor(x.grid_host[c] * (double)budget[bh / bp.Hkv] + 0.5);
      pl.counts[(size_t)c * BH + bh] = r;
      if (r > pl.r_max[bh]) pl.r_max[bh] = r;
    }
  std::vector<HeadMeta> hm;
  for (int c = 0; c < pl.NG; ++c) {
    head_meta(bp, seq_len, budget, pl.counts.data() + (size_t)c * BH, p.recent_window, hm);
    if (!fold_build_plan(hm, &bp)) return false;
  }
  if (!layout_build_plan(&bp)) return false;
  pl.dec_full = make_decode_plan(full_shape(pl));
  pl.dec_cand = make_decode_plan(cand_shape(pl));
  for (const DecodePlan* d : {&pl.dec_full, &pl.dec_cand})
    if ((size_t)d->GP * d->P * sizeof(float) > decode_max_lds_weights()) return false;
  const size_t NGB = (size_t)pl.NG * BH;  // candidate (b, kv head) pairs
  const size_t esz = bp.dtype == RESKV_BF16 ? 2 : 4;
  const size_t qrows = (size_t)bp.Hkv * pl.GC;  // decode query heads per sequence
  size_t off = bp.bytes;
  auto take = [&](size_t bytes) { const size_t o = off; off = align_up(off + bytes, 256); return o; };
  pl.off_meta = take((NGB + BH) * sizeof(HeadMeta));
  pl.off_kc = take(NGB * bp.C * bp.D * esz);
  pl.off_vc = take(NGB * bp.C * bp.D * esz);
  pl.off_logc = take(NGB * bp.Rcap * sizeof(float));
  pl.off_midx = take(NGB * bp.C * sizeof(int32_t));
  pl.off_rlen = take(NGB * sizeof(int32_t));
  pl.off_mlen = take(NGB * sizeof(int32_t));
  pl.off_rlen0 = take(BH * sizeof(int32_t));
  pl.off_mlen0 = take(BH * sizeof(int32_t));
  pl.off_logc0 = take(BH * sizeof(float));
  pl.off_q = take((size_t)pl.NQC * pl.NG * bp.B * qrows * bp.D * esz);
  pl.off_out_full = take((size_t)pl.NQC * bp.B * qrows * bp.D * sizeof(float));
  pl.off_out_cand = take((size_t)pl.NQC * pl.NG * bp.B * qrows * bp.D * sizeof(float));
  pl.off_dec = take(pl.dec_full.bytes > pl.dec_cand.bytes ? pl.dec_full.bytes : pl.dec_cand.bytes);
  pl.off_loss = take(NGB * sizeof(float));
  pl.off_choice = take(BH * sizeof(int32_t));
  pl.bytes = off;
  return true;
}

hipError_t launch_build_proxy(const reskv_shape_t& s, const reskv_build_params_t& p,
                              const reskv_proxy_params_t& x, const reskv_gate_t& g, const ProxyPlan& pl,
                              const void* k, const void* v, const int32_t* seq_len, const void* q_obs,
                              const int32_t* budget, void* kc, void* vc, float* logc, int32_t* main_idx,
                              int32_t* res_len, int32_t* main_len, float* val_loss, void* workspace,
                              hipStream_t stream) {
  (void)s;
  const BuildPlan& bp = pl.build;
  char* ws = static_cast<char*>(workspace);
  const int BH = bp.B * bp.Hkv;
  const size_t esz = bp.dtype == RESKV_BF16 ? 2 : 4;
  HeadMeta* cmeta = reinterpret_cast<HeadMeta*>(ws + pl.off_meta);  // [NG][BH], then the scoring sizes
  HeadMeta* smeta = cmeta + (size_t)pl.NG * BH;
  char* kc_c = ws + pl.off_kc;
  char* vc_c = ws + pl.off_vc;
  float* logc_c = reinterpret_cast<float*>(ws + pl.off_logc);
  int32_t* midx_c = reinterpret_cast<int32_t*>(ws + pl.off_midx);
  int32_t* rlen_c = reinterpret_cast<int32_t*>(ws + pl.off_rlen);
  int32_t* mlen_c = reinterpret_cast<int32_t*>(ws + pl.off_mlen);
  hipError_t e;
#define RESKV_TRY(expr) do { e = (expr); if (e != hipSuccess) return e; } while (0)
  for (int c = 0; c < pl.NG; ++c)
    RESKV_TRY(upload_meta(bp, seq_len, budget, pl.counts.data() + (size_t)c * BH, p.recent_window,
                          cmeta + (size_t)c * BH, stream));
  RESKV_TRY(upload_meta(bp, seq_len, budget, pl.r_max.data(), p.recent_window, smeta, stream));
  // scoring once with the fit rows; the build scratch sits at the start of the workspace
  RESKV_TRY(launch_build_scores(bp, k, q_obs, smeta, workspace, stream));
  const size_t cache_elems = (size_t)BH * bp.C * bp.D;  // elements of one candidate's kc
  for (int c = 0; c < pl.NG; ++c) {
    const BuildOut out{kc_c + c * cache_elems * esz, vc_c + c * cache_elems * esz,
                       logc_c + (size_t)c * BH * bp.Rcap, midx_c + (size_t)c * BH * bp.C,
                       rlen_c + (size_t)c * BH, mlen_c + (size_t)c * BH};
    RESKV_TRY(launch_build_candidate(bp, k, v, cmeta + (size_t)c * BH, out, nullptr, nullptr, nullptr, workspace, stream));
  }
  // validation queries and the uncompressed reference lengths
  GatherArgs ga{q_obs, ws + pl.off_q, bp.B, bp.Hq, bp.Hkv, bp.G, bp.w, bp.wr, pl.val, pl.GV, pl.GC, pl.NQC, pl.NG};
  CopyArgs ca{cmeta, reinterpret_cast<int32_t*>(ws + pl.off_choice), kc_c, vc_c, logc_c, midx_c,
              kc, vc, logc, main_idx, bp.B, bp.Hkv, bp.C, bp.Rcap};
  RESKV_TRY(launch_tail(pl, ga, ca, stream, 0));
  int32_t* rlen0 = reinterpret_cast<int32_t*>(ws + pl.off_rlen0);
  int32_t* mlen0 = reinterpret_cast<int32_t*>(ws + pl.off_mlen0);
  float* logc0 = reinterpret_cast<float*>(ws + pl.off_logc0);
  hipLaunchKernelGGL(proxy_full_lengths, dim3((BH + kThreads - 1) / kThreads), dim3(kThreads), 0, stream, smeta,
                     rlen0, mlen0, logc0, BH);
  RESKV_TRY(hipGetLastError());
  // decode: the gate's scalar threshold applies to every validation query
  reskv_gate_t gs = g;
  gs.tau = nullptr;
  const reskv_shape_t sf = full_shape(pl), sc = cand_shape(pl);
  const size_t qrows = (size_t)bp.Hkv * pl.GC;
  float* out_full = reinterpret_cast<float*>(ws + pl.off_out_full);
  float* out_cand = reinterpret_cast<float*>(ws + pl.off_out_cand);
  for (int ch = 0; ch < pl.NQC; ++ch) {
    const char* qch = ws + pl.off_q + (size_t)ch * pl.NG * bp.B * qrows * bp.D * esz;
    RESKV_TRY(launch_decode(sf, gs, pl.dec_full, qch, const_cast<void*>(k), const_cast<void*>(v), logc0, rlen0,
                            mlen0, nullptr, nullptr, out_full + (size_t)ch * bp.B * qrows * bp.D, nullptr, nullptr,
                            nullptr, ws + pl.off_dec, stream));
    RESKV_TRY(launch_decode(sc, gs, pl.dec_cand, qch, kc_c, vc_c, logc_c, rlen_c, mlen_c, nullptr, nullptr,
                            out_cand + (size_t)ch * pl.NG * bp.B * qrows * bp.D, nullptr, nullptr, nullptr,
                            ws + pl.off_dec, stream));
  }
  float* loss = reinterpret_cast<float*>(ws + pl.off_loss);
  hipLaunchKernelGGL(proxy_loss, dim3(BH, pl.NG), dim3(kThreads), 0, stream, out_full, out_cand, loss, bp.B, bp.Hkv,
                     pl.GC, pl.GV, pl.NQC, pl.NG, bp.D);
  RESKV_TRY(hipGetLastError());
  hipLaunchKernelGGL(proxy_choose, dim3((BH + kThreads - 1) / kThreads), dim3(kThreads), 0, stream, cmeta, loss,
                     x.delta, pl.NG, BH, reinterpret_cast<int32_t*>(ws + pl.off_choice), res_len, main_len, val_loss);
  RESKV_TRY(hipGetLastError());
  RESKV_TRY(launch_tail(pl, ga, ca, stream, 1));
#undef RESKV_TRY
  return hipSuccess;
}

}  // namespace reskv
