// Shared-softmax residual decode (Sec. 5.4; Sec. 5.5.2 gate; App. D, Algorithm 2).
//
// Split-K flash decode over the fixed-budget cache of one layer:
//   decode_split   one block = 256 slots of one (b, kv head), all of one kind
//                  (residual slots [0, r) or main slots [r, r+n)); it writes the
//                  block's partial (running max m, sum l, unnormalised acc) per
//                  query head of the group. Logits are kept in base 2
//                  (log2(e)/sqrt(d) folded into one scale).
//   decode_combine one block per (b, kv head): merges the main partials, takes
//                  p_max = 1 / l_main (the max term contributes exactly 1),
//                  evaluates the gate, shifts the residual partials by log g and
//                  normalises main and residual under one denominator.
//
// Work split inside decode_split: 4 waves x 64 slots. Q.K^T runs on MFMA
// (16 heads x 16 slots per tile; 16x16x32 bf16 or 16x16x4 f32), each lane
// fetching one quarter of a key row with 16-byte loads. The softmax max/sum is
// a 16-lane butterfly; probabilities go through LDS to the P.V stage, which
// streams value rows with 16-byte loads and accumulates in fp32 registers.
#include "common.h"
#include "internal.h"

namespace reskv {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kWaveSlots = 64;
constexpr int kTiles = kWaveSlots / 16;
static_assert(kWaves * kWaveSlots == kDecChunk, "chunk = waves x wave slots");

struct SplitArgs {
  const void* q;
  const void* kc;
  const void* vc;
  const float* logc;
  const int32_t* res_len;
  const int32_t* main_len;
  float* part_acc;  // [B*Hkv][P][GP][D]
  float* part_ml;   // [B*Hkv][P][GP][2]  (m in base 2, l)
  int Hq, Hkv, G, C, Rcap, PR, P;
  float qk_scale;   // log2(e) / sqrt(d)
  float beta_log2;  // beta * log2(e)
};

struct CombineArgs {
  const float* part_acc;
  const float* part_ml;
  const int32_t* res_len;
  const int32_t* main_len;
  const float* tau;
  float tau_scalar, alpha, g_min;
  float* out;
  float* dbg_lse_main;
  float* dbg_lse_res;
  float* dbg_gate;
  int Hq, Hkv, G, C, Rcap, PR, P;
};

__device__ __forceinline__ void cache_lengths(const int32_t* res_len, const int32_t* main_len,
                                              int bh, int C, int Rcap, int& r, int& n) {
  r = clampi(res_len[bh], 0, min(Rcap, C));
  n = clampi(main_len[bh], 0, C - r);
}

// ---- Q.K^T on MFMA: C[head][slot] for 16 heads x 16 slots ------------------
// Lane (col + 16*grp): A operand = query head `col`, B operand = key row of
// slot `col`; lane group `grp` owns the contiguous quarter
// [grp*D/4, (grp+1)*D/4) of the head dimension for both operands.
template <typename T, int D>
struct QKTile;

template <int D>
struct QKTile<uint16_t, D> {
  static constexpr int kSteps = D / 32;  // 16x16x32 bf16 steps per quarter row
  bf16x8_t q[kSteps];
  __device__ void load_q(const uint16_t* qrow, bool live) {
#pragma unroll
    for (int i = 0; i < kSteps; ++i) {
      uint4 w = live ? *reinterpret_cast<const uint4*>(qrow + 8 * i) : make_uint4(0, 0, 0, 0);
      q[i] = as_bf16x8(w);
    }
  }
  __device__ f32x4_t run(const uint16_t* krow) const {
    uint4 k[kSteps];
#pragma unroll
    for (int i = 0; i < kSteps; ++i) k[i] = *reinterpret_cast<const uint4*>(krow + 8 * i);
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < kSteps; ++i)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(q[i], as_bf16x8(k[i]), acc, 0, 0, 0);
    return acc;
  }
};

template <int D>
struct QKTile<float, D> {
  static constexpr int kSteps = D / 4;  // 16x16x4 f32 steps per quarter row
  float q[kSteps];
  __device__ void load_q(const float* qrow, bool live) {
#pragma unroll
    for (int i = 0; i < kSteps; i += 4) {
      float4 w = live ? *reinterpret_cast<const float4*>(qrow + i) : make_float4(0.f, 0.f, 0.f, 0.f);
      q[i] = w.x; q[i + 1] = w.y; q[i + 2] = w.z; q[i + 3] = w.w;
    }
  }
  __device__ f32x4_t run(const float* krow) const {
    float k[kSteps];
#pragma unroll
    for (int i = 0; i < kSteps; i += 4) {
      float4 w = *reinterpret_cast<const float4*>(krow + i);
      k[i] = w.x; k[i + 1] = w.y; k[i + 2] = w.z; k[i + 3] = w.w;
    }
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < kSteps; ++i) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q[i], k[i], acc, 0, 0, 0);
    return acc;
  }
};

template <typename T, int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_split(SplitArgs a) {
  const int p = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  int r, n;
  cache_lengths(a.res_len, a.main_len, bh, a.C, a.Rcap, r, n);
  const bool is_res = p < a.PR;
  int lo, hi;
  if (is_res) {
    lo = p * kDecChunk;
    hi = min(lo + kDecChunk, r);
  } else {
    lo = r + (p - a.PR) * kDecChunk;
    hi = min(lo + kDecChunk, r + n);
  }
  if (lo >= hi) return;  // block-uniform

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int w_lo = lo + wave * kWaveSlots;
  const int nvalid = min(w_lo + kWaveSlots, hi) - w_lo;  // wave-uniform, may be <= 0

  __shared__ float s_p[kWaves][kWaveSlots][GP];
  __shared__ float s_acc[kWaves][GP][D];
  __shared__ float s_m[kWaves][GP];
  __shared__ float s_l[kWaves][GP];

  const T* kc = static_cast<const T*>(a.kc) + (size_t)bh * a.C * D;
  const T* vc = static_cast<const T*>(a.vc) + (size_t)bh * a.C * D;

  float mrow[4], lrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { mrow[i] = kNegInf; lrow[i] = 0.f; }

  if (nvalid > 0) {
    QKTile<T, D> qk;
    const T* qrow = static_cast<const T*>(a.q) + ((size_t)b * a.Hq + (size_t)kvh * a.G + col) * D + grp * (D / 4);
    qk.load_q(qrow, col < a.G);

    f32x4_t s[kTiles];
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
      const int slot = w_lo + 16 * t + col;
      const int row = (16 * t + col < nvalid) ? slot : w_lo;
      s[t] = qk.run(kc + (size_t)row * D + grp * (D / 4));
    }
    // scale to base-2 logits, add beta*log c for residual entries, mask the tail
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
      const bool live = 16 * t + col < nvalid;
      float lc = 0.f;
      if (is_res && live) lc = a.logc[(size_t)bh * a.Rcap + w_lo + 16 * t + col];
      const bool dead = !live || (is_res && lc == kNegInf);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v = s[t][i] * a.qk_scale;
        if (is_res) v += a.beta_log2 * lc;
        s[t][i] = dead ? kNegInf : v;
      }
    }
    // per-head max and sum over the wave's slots (16-lane butterflies)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float m = s[0][i];
#pragma unroll
      for (int t = 1; t < kTiles; ++t) m = fmaxf(m, s[t][i]);
      m = wave_xor_max(m, 1); m = wave_xor_max(m, 2);
      m = wave_xor_max(m, 4); m = wave_xor_max(m, 8);
      mrow[i] = m;
      const float mu = (m == kNegInf) ? 0.f : m;
      float l = 0.f;
#pragma unroll
      for (int t = 0; t < kTiles; ++t) {
        const float e = exp2f(s[t][i] - mu);
        s[t][i] = e;
        l += e;
      }
      l = wave_xor_add(l, 1); l = wave_xor_add(l, 2);
      l = wave_xor_add(l, 4); l = wave_xor_add(l, 8);
      lrow[i] = l;
    }
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int h = 4 * grp + i;
        if (h < GP) s_p[wave][16 * t + col][h] = s[t][i];
      }
    }
  }
  __syncthreads();

  // P.V: lane = (chunk c of 8 columns, row phase ph)
  constexpr int CPR = D / 8;
  constexpr int RP = 64 / CPR;
  const int c = lane % CPR, ph = lane / CPR;
  float acc[GP][8];
#pragma unroll
  for (int h = 0; h < GP; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
  if (nvalid > 0) {
    const T* vbase = vc + (size_t)w_lo * D + 8 * c;
    for (int j = ph; j < nvalid; j += RP) {
      float v[8];
      load8_f32(vbase + (size_t)j * D, v);
      float pr[GP];
#pragma unroll
      for (int h = 0; h < GP; ++h) pr[h] = s_p[wave][j][h];
#pragma unroll
      for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pr[h], v[e], acc[h][e]);
    }
  }
#pragma unroll
  for (int msk = CPR; msk < 64; msk <<= 1)
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = wave_xor_add(acc[h][e], msk);
  if (ph == 0) {
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) s_acc[wave][h][8 * c + e] = acc[h][e];
  }
  if (col == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * grp + i;
      if (h < GP) {
        s_m[wave][h] = nvalid > 0 ? mrow[i] : kNegInf;
        s_l[wave][h] = nvalid > 0 ? lrow[i] : 0.f;
      }
    }
  }
  __syncthreads();

  // merge the 4 waves into the block's partial
  const size_t pbase = ((size_t)bh * a.P + p) * GP;
  for (int idx = tid; idx < GP * D; idx += kThreads) {
    const int h = idx / D, d = idx % D;
    float M = s_m[0][h];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) M = fmaxf(M, s_m[w][h]);
    float o = 0.f, l = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float f = exp2f(s_m[w][h] - M);
        o = fmaf(f, s_acc[w][h][d], o);
        l = fmaf(f, s_l[w][h], l);
      }
    }
    a.part_acc[(pbase + h) * D + d] = o;
    if (d == 0) {
      a.part_ml[(pbase + h) * 2 + 0] = M;
      a.part_ml[(pbase + h) * 2 + 1] = l;
    }
  }
}

template <int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_combine(CombineArgs a) {
  const int kvh = blockIdx.x, b = blockIdx.y;
  const int bh = b * a.Hkv + kvh;
  int r, n;
  cache_lengths(a.res_len, a.main_len, bh, a.C, a.Rcap, r, n);
  const int nRC = (r + kDecChunk - 1) / kDecChunk;
  const int nMC = (n + kDecChunk - 1) / kDecChunk;
  const float* ml = a.part_ml + (size_t)bh * a.P * GP * 2;
  const float* pacc = a.part_acc + (size_t)bh * a.P * GP * D;

  __shared__ float s_mx[GP], s_lg2g[GP], s_inv[GP];
  const int tid = threadIdx.x;
  if (tid < a.G) {
    const int h = tid;
    float mM = kNegInf, mR = kNegInf;
    for (int q = 0; q < nMC; ++q) mM = fmaxf(mM, ml[((a.PR + q) * GP + h) * 2]);
    for (int q = 0; q < nRC; ++q) mR = fmaxf(mR, ml[(q * GP + h) * 2]);
    float lM = 0.f, lR = 0.f;
    if (mM != kNegInf)
      for (int q = 0; q < nMC; ++q) {
        const float* e = ml + ((a.PR + q) * GP + h) * 2;
        lM = fmaf(e[1], exp2f(e[0] - mM), lM);
      }
    if (mR != kNegInf)
      for (int q = 0; q < nRC; ++q) {
        const float* e = ml + (q * GP + h) * 2;
        lR = fmaf(e[1], exp2f(e[0] - mR), lR);
      }
    // p_max = max_p e^{a_p} / sum_p e^{a_p} = 1 / lM (the max term is exactly 1)
    const float pmax = lM > 0.f ? 1.f / lM : 1.f;
    const int qh = b * a.Hq + kvh * a.G + h;
    const float tau = a.tau ? a.tau[qh] : a.tau_scalar;
    const float g = fmaxf(a.g_min, 1.f / (1.f + expf(-(tau - pmax) * a.alpha)));
    const float lg2g = g > 0.f ? log2f(g) : kNegInf;
    const float mRg = (mR == kNegInf || lg2g == kNegInf) ? kNegInf : mR + lg2g;
    const float Mx = fmaxf(mM, mRg);
    float den = 0.f;
    if (mM != kNegInf) den += lM * exp2f(mM - Mx);
    if (mRg != kNegInf) den += lR * exp2f(mRg - Mx);
    s_mx[h] = Mx;
    s_lg2g[h] = lg2g;
    s_inv[h] = den > 0.f ? 1.f / den : 0.f;
    if (a.dbg_lse_main) a.dbg_lse_main[qh] = lM > 0.f ? (mM + log2f(lM)) * kLn2 : kNegInf;
    if (a.dbg_lse_res) a.dbg_lse_res[qh] = lR > 0.f ? (mR + log2f(lR)) * kLn2 : kNegInf;
    if (a.dbg_gate) a.dbg_gate[qh] = g;
  }
  __syncthreads();
  for (int idx = tid; idx < a.G * D; idx += kThreads) {
    const int h = idx / D, d = idx % D;
    const float Mx = s_mx[h], lg2g = s_lg2g[h];
    float o = 0.f;
    for (int q = 0; q < nMC; ++q) {
      const int pp = a.PR + q;
      const float m = ml[(pp * GP + h) * 2];
      if (m != kNegInf) o = fmaf(exp2f(m - Mx), pacc[(pp * GP + h) * D + d], o);
    }
    if (lg2g != kNegInf)
      for (int q = 0; q < nRC; ++q) {
        const float m = ml[(q * GP + h) * 2];
        if (m != kNegInf) o = fmaf(exp2f(m + lg2g - Mx), pacc[(q * GP + h) * D + d], o);
      }
    a.out[((size_t)b * a.Hq + kvh * a.G + h) * D + d] = o * s_inv[h];
  }
}

template <typename T, int D>
__global__ void append_kernel(const T* k_new, const T* v_new, T* kc, T* vc, const int32_t* res_len,
                              int32_t* main_len, int C) {
  const int bh = blockIdx.x;
  const int r = clampi(res_len[bh], 0, C);
  const int n = clampi(main_len[bh], 0, C - r);
  __syncthreads();
  if (r + n >= C) return;  // block-uniform: the cache is full
  const size_t slot = (size_t)bh * C + r + n;
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    kc[slot * D + d] = k_new[(size_t)bh * D + d];
    vc[slot * D + d] = v_new[(size_t)bh * D + d];
  }
  __syncthreads();
  if (threadIdx.x == 0) main_len[bh] = n + 1;
}

template <typename T, int D, int GP>
hipError_t launch_typed(const DecodePlan& pl, const SplitArgs& sa, const CombineArgs& ca,
                        hipStream_t stream) {
  dim3 g1(pl.P, pl.Hkv, pl.B);
  hipLaunchKernelGGL((decode_split<T, D, GP>), g1, dim3(kThreads), 0, stream, sa);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 g2(pl.Hkv, pl.B);
  hipLaunchKernelGGL((decode_combine<D, GP>), g2, dim3(kThreads), 0, stream, ca);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_gp(const DecodePlan& pl, const SplitArgs& sa, const CombineArgs& ca,
                     hipStream_t stream) {
  switch (pl.GP) {
    case 1: return launch_typed<T, D, 1>(pl, sa, ca, stream);
    case 2: return launch_typed<T, D, 2>(pl, sa, ca, stream);
    case 4: return launch_typed<T, D, 4>(pl, sa, ca, stream);
    case 8: return launch_typed<T, D, 8>(pl, sa, ca, stream);
    case 16: return launch_typed<T, D, 16>(pl, sa, ca, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace

DecodePlan make_decode_plan(const reskv_shape_t& s) {
  DecodePlan p{};
  p.B = s.batch; p.Hq = s.num_q_heads; p.Hkv = s.num_kv_heads;
  p.G = s.num_q_heads / s.num_kv_heads;
  p.GP = p.G <= 1 ? 1 : p.G <= 2 ? 2 : p.G <= 4 ? 4 : p.G <= 8 ? 8 : 16;
  p.D = s.head_dim; p.C = s.slot_cap; p.Rcap = s.res_cap;
  const int rmax = s.res_cap < s.slot_cap ? s.res_cap : s.slot_cap;
  p.PR = (rmax + kDecChunk - 1) / kDecChunk;
  p.PM = (s.slot_cap + kDecChunk - 1) / kDecChunk;
  p.P = p.PR + p.PM;
  const size_t units = (size_t)p.B * p.Hkv * p.P * p.GP;
  p.acc_off = 0;
  p.ml_off = align_up(units * p.D * sizeof(float), 256);
  p.bytes = p.ml_off + align_up(units * 2 * sizeof(float), 256);
  return p;
}

hipError_t launch_decode(const reskv_shape_t& s, const reskv_gate_t& g, const DecodePlan& pl,
                         const void* q, const void* kc, const void* vc, const float* logc,
                         const int32_t* res_len, const int32_t* main_len, float* out,
                         float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate,
                         void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  SplitArgs sa{};
  sa.q = q; sa.kc = kc; sa.vc = vc; sa.logc = logc;
  sa.res_len = res_len; sa.main_len = main_len;
  sa.part_acc = reinterpret_cast<float*>(ws + pl.acc_off);
  sa.part_ml = reinterpret_cast<float*>(ws + pl.ml_off);
  sa.Hq = pl.Hq; sa.Hkv = pl.Hkv; sa.G = pl.G; sa.C = pl.C; sa.Rcap = pl.Rcap;
  sa.PR = pl.PR; sa.P = pl.P;
  sa.qk_scale = kLog2e / sqrtf((float)pl.D);
  sa.beta_log2 = g.beta * kLog2e;
  CombineArgs ca{};
  ca.part_acc = sa.part_acc; ca.part_ml = sa.part_ml;
  ca.res_len = res_len; ca.main_len = main_len;
  ca.tau = g.tau; ca.tau_scalar = g.tau_scalar; ca.alpha = g.alpha; ca.g_min = g.g_min;
  ca.out = out; ca.dbg_lse_main = dbg_lse_main; ca.dbg_lse_res = dbg_lse_res; ca.dbg_gate = dbg_gate;
  ca.Hq = pl.Hq; ca.Hkv = pl.Hkv; ca.G = pl.G; ca.C = pl.C; ca.Rcap = pl.Rcap;
  ca.PR = pl.PR; ca.P = pl.P;
  const bool bf = s.dtype == RESKV_BF16;
  if (pl.D == 128) return bf ? launch_gp<uint16_t, 128>(pl, sa, ca, stream) : launch_gp<float, 128>(pl, sa, ca, stream);
  if (pl.D == 64) return bf ? launch_gp<uint16_t, 64>(pl, sa, ca, stream) : launch_gp<float, 64>(pl, sa, ca, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_append(const reskv_shape_t& s, const void* k_new, const void* v_new, void* kc,
                         void* vc, const int32_t* res_len, int32_t* main_len, hipStream_t stream) {
  dim3 grid(s.batch * s.num_kv_heads);
  const int C = s.slot_cap;
  if (s.dtype == RESKV_BF16) {
    if (s.head_dim == 128)
      hipLaunchKernelGGL((append_kernel<uint16_t, 128>), grid, dim3(128), 0, stream,
                         (const uint16_t*)k_new, (const uint16_t*)v_new, (uint16_t*)kc, (uint16_t*)vc, res_len, main_len, C);
    else
      hipLaunchKernelGGL((append_kernel<uint16_t, 64>), grid, dim3(64), 0, stream,
                         (const uint16_t*)k_new, (const uint16_t*)v_new, (uint16_t*)kc, (uint16_t*)vc, res_len, main_len, C);
  } else {
    if (s.head_dim == 128)
      hipLaunchKernelGGL((append_kernel<float, 128>), grid, dim3(128), 0, stream,
                         (const float*)k_new, (const float*)v_new, (float*)kc, (float*)vc, res_len, main_len, C);
    else
      hipLaunchKernelGGL((append_kernel<float, 64>), grid, dim3(64), 0, stream,
                         (const float*)k_new, (const float*)v_new, (float*)kc, (float*)vc, res_len, main_len, C);
  }
  return hipGetLastError();
}

}  // namespace reskv
