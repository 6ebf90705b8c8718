// Shared-softmax residual decode (Sec. 5.4; Sec. 5.5.2 gate; App. D, Algorithm 2).
//
// Split-K flash decode over the fixed-budget cache of one layer, in two
// launches:
//   decode_split   one block = 256 slots of one (b, kv head), all of one kind
//                  (residual slots [0, r) or main slots [r, r+n)), one 64-slot
//                  unit per wave; it writes the block's partial record (max
//                  m, sum l, unnormalised acc) per query head of the group.
//                  Logits are kept in base 2, with log2(e)/sqrt(d) folded
//                  into one scale.
//   decode_combine one block per (b, kv head): the main records give
//                  p_max = 1 / l_main (the max term contributes exactly 1),
//                  the gate follows, the residual records are shifted by
//                  log g, and main and residual share one denominator.
// The combine is a separate launch rather than a last-arriving-block epilogue:
// on this multi-XCD part a device-scope release/acquire per block writes back
// and invalidates L2, which costs far more than one more launch.
//
// Per unit: Q.K^T on MFMA (16 heads x 16 slots per tile; 16x16x32 bf16 or
// 16x16x4 f32), each lane fetching one quarter of a key row with 16-byte
// loads; the per-head max/sum is a 16-lane butterfly; probabilities and the
// rescale factors pass through LDS (wave-private rows) to the P.V stage, which
// widens 16-byte value loads and accumulates in fp32 registers.
#include "common.h"
#include "internal.h"

namespace reskv {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kUnit = 64;              // slots per wave unit
constexpr int kTiles = kUnit / 16;     // MFMA tiles per unit
constexpr int kChunk = kWaves * kUnit; // slots per split block
constexpr int kWholeHeadMin = 256;     // (b, kv head) pairs that fill the 256 CUs

struct DecodeArgs {
  const void* q;
  const void* kc;
  const void* vc;
  const float* logc;
  const int32_t* res_len;
  int32_t* main_len;
  const void* k_new;  // fused append (decode_head only), or NULL
  const void* v_new;
  float* part_acc;  // [B*Hkv][P][GP][D]
  float* part_ml;   // [B*Hkv][P][GP][2]  (m in base 2, l)
  const float* tau;
  float* out;
  float* dbg_lse_main;
  float* dbg_lse_res;
  float* dbg_gate;
  int Hq, Hkv, G, C, Rcap, PR, P;
  float qk_scale;   // log2(e) / sqrt(d)
  float beta_log2;  // beta * log2(e)
  float tau_scalar, alpha, g_min;
};

__device__ __forceinline__ void cache_lengths(const int32_t* res_len, const int32_t* main_len,
                                              int bh, int C, int Rcap, int& r, int& n) {
  r = clampi(res_len[bh], 0, min(Rcap, C));
  n = clampi(main_len[bh], 0, C - r);
}

// ---- Q.K^T on MFMA: C[head][slot] for 16 heads x 16 slots ------------------
// A operand = query head (lane % 16), B operand = key row of slot (lane % 16).
template <typename T, int D>
struct QK {
  using KFrag = Frag<T, D>;
  Frag<T, D> q;
  __device__ void load_q(const T* qrow, bool live) {
    if (live) q.load(qrow); else q.zero();
  }
  __device__ static void load_k(KFrag& f, const T* krow) { f.load(krow); }
  __device__ f32x4_t run(const KFrag& f) const { return mma<D>(q, f, zero4()); }
};

// 8 consecutive value-row elements, loaded raw and widened later.
template <typename T>
struct VRow;
template <>
struct VRow<uint16_t> {
  uint4 w;
  __device__ void load(const uint16_t* p) { w = *reinterpret_cast<const uint4*>(p); }
  __device__ void widen(float (&x)[8]) const {
    x[0] = bf16_lo(w.x); x[1] = bf16_hi(w.x); x[2] = bf16_lo(w.y); x[3] = bf16_hi(w.y);
    x[4] = bf16_lo(w.z); x[5] = bf16_hi(w.z); x[6] = bf16_lo(w.w); x[7] = bf16_hi(w.w);
  }
};
template <>
struct VRow<float> {
  float4 a, b;
  __device__ void load(const float* p) {
    a = *reinterpret_cast<const float4*>(p);
    b = *reinterpret_cast<const float4*>(p + 4);
  }
  __device__ void widen(float (&x)[8]) const {
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
};


// Raw loads of one 64-slot unit for one lane: key fragments (+ log-counts)
// and value-row chunks.
template <typename T, int D>
struct KRegs {
  typename QK<T, D>::KFrag k[kTiles];
  float lc[kTiles];
};
template <typename T, int D>
struct VRegs {
  static constexpr int CPR = D / 8;         // 8-column chunks per value row
  static constexpr int RP = 64 / CPR;       // rows covered by one wave-wide load
  static constexpr int NR = kUnit / RP;     // value rows per lane
  VRow<T> v[NR];
};

// Loads of unit [s0, s0 + nvalid); rows past the tail are clamped to the
// unit's first row (their probabilities are zero).
template <typename T, int D>
__device__ __forceinline__ void load_unit_k(KRegs<T, D>& u, const T* kc, const float* logc, bool is_res, int s0,
                                            int nvalid, int col, int grp) {
#pragma unroll
  for (int t = 0; t < kTiles; ++t) {
    const int row = (16 * t + col < nvalid) ? s0 + 16 * t + col : s0;
    QK<T, D>::load_k(u.k[t], kc + (size_t)row * D + grp * (D / 4));
  }
#pragma unroll
  for (int t = 0; t < kTiles; ++t)
    u.lc[t] = (is_res && 16 * t + col < nvalid) ? logc[s0 + 16 * t + col] : 0.f;
}

template <typename T, int D>
__device__ __forceinline__ void load_unit_v(VRegs<T, D>& u, const T* vc, int s0, int nvalid, int c, int ph) {
#pragma unroll
  for (int k = 0; k < VRegs<T, D>::NR; ++k) {
    const int j = ph + VRegs<T, D>::RP * k;
    u.v[k].load(vc + (size_t)(s0 + min(j, nvalid - 1)) * D + 8 * c);
  }
}

// Online-softmax state of one wave for one kind.
template <int GP>
struct WaveState {
  float m[4], l[4];   // per head 4*grp + i (replicated over the 16 lanes of a group)
  float acc[GP][8];   // per head, 8 columns of this lane's chunk, this lane's row phase
  __device__ void reset() {
#pragma unroll
    for (int i = 0; i < 4; ++i) { m[i] = kNegInf; l[i] = 0.f; }
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
  }
};

// One unit: logits on MFMA, then (once the key fragments are consumed) the
// value loads, then the online softmax update and P.V.
template <typename T, int D, int GP>
__device__ __forceinline__ void process_unit(const KRegs<T, D>& u, VRegs<T, D>& vr, const QK<T, D>& qk,
                                             WaveState<GP>& st, float (*s_p)[GP], float* s_alpha, bool is_res,
                                             int nvalid, float qk_scale, float beta_log2, int col, int grp, int c,
                                             int ph, const T* vc, int s0) {
  f32x4_t s[kTiles];
#pragma unroll
  for (int t = 0; t < kTiles; ++t) s[t] = qk.run(u.k[t]);
  load_unit_v<T, D>(vr, vc, s0, nvalid, c, ph);
#pragma unroll
  for (int t = 0; t < kTiles; ++t) {
    const bool live = 16 * t + col < nvalid;
    const bool dead = !live || (is_res && u.lc[t] == kNegInf);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = s[t][i] * qk_scale;
      if (is_res) v += beta_log2 * u.lc[t];
      s[t][i] = dead ? kNegInf : v;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float m = s[0][i];
#pragma unroll
    for (int t = 1; t < kTiles; ++t) m = fmaxf(m, s[t][i]);
    m = wave_xor_max(m, 1); m = wave_xor_max(m, 2);
    m = wave_xor_max(m, 4); m = wave_xor_max(m, 8);
    const float m_new = fmaxf(st.m[i], m);
    const float mu = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = exp2f(st.m[i] - mu);
    float l = 0.f;
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
      const float e = exp2f(s[t][i] - mu);
      s[t][i] = e;
      l += e;
    }
    l = wave_xor_add(l, 1); l = wave_xor_add(l, 2);
    l = wave_xor_add(l, 4); l = wave_xor_add(l, 8);
    st.l[i] = fmaf(st.l[i], alpha, l);
    st.m[i] = m_new;
    const int h = 4 * grp + i;
    if (h < GP && col == 0) s_alpha[h] = alpha;
  }
#pragma unroll
  for (int t = 0; t < kTiles; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * grp + i;
      if (h < GP) s_p[16 * t + col][h] = s[t][i];
    }
  // LDS traffic of one wave executes in order; this keeps the compiler from
  // moving the reads below above the writes
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  float al[GP];
#pragma unroll
  for (int h = 0; h < GP; ++h) al[h] = s_alpha[h];
#pragma unroll
  for (int h = 0; h < GP; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) st.acc[h][e] *= al[h];
#pragma unroll
  for (int k = 0; k < VRegs<T, D>::NR; ++k) {
    const int j = ph + VRegs<T, D>::RP * k;
    float v[8];
    vr.v[k].widen(v);
    float pr[GP];
#pragma unroll
    for (int h = 0; h < GP; ++h) pr[h] = s_p[j][h];
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) st.acc[h][e] = fmaf(pr[h], v[e], st.acc[h][e]);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <typename T, int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_split(DecodeArgs a) {
  using Regs = VRegs<T, D>;
  const int p = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  int r, n;
  cache_lengths(a.res_len, a.main_len, bh, a.C, a.Rcap, r, n);
  // block p < PR covers residual slots [256p, 256p + 256) of [0, r); block
  // p >= PR covers main slots [r + 256(p-PR), ...) of [r, r + n)
  const bool is_res = p < a.PR;
  const int base = is_res ? 0 : r;
  const int end = is_res ? r : r + n;
  const int lo = base + (is_res ? p : p - a.PR) * kChunk;
  if (lo >= end) return;  // block-uniform

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int c = lane % Regs::CPR, ph = lane / Regs::CPR;

  __shared__ float s_p[kWaves][kUnit][GP];
  __shared__ float s_alpha[kWaves][GP];
  __shared__ float s_acc[kWaves][GP][D];
  __shared__ float s_m[kWaves][GP];
  __shared__ float s_l[kWaves][GP];

  const T* kc = static_cast<const T*>(a.kc) + (size_t)bh * a.C * D;
  const T* vc = static_cast<const T*>(a.vc) + (size_t)bh * a.C * D;
  const float* logc = a.logc + (size_t)bh * a.Rcap;

  WaveState<GP> st;
  st.reset();
  const int s0 = lo + wave * kUnit;
  if (s0 < end) {  // wave-uniform
    QK<T, D> qk;
    qk.load_q(static_cast<const T*>(a.q) + ((size_t)b * a.Hq + (size_t)kvh * a.G + col) * D + grp * (D / 4),
              col < a.G);
    KRegs<T, D> kr;
    VRegs<T, D> vr;
    const int nvalid = min(kUnit, end - s0);
    load_unit_k<T, D>(kr, kc, logc, is_res, s0, nvalid, col, grp);
    process_unit<T, D, GP>(kr, vr, qk, st, s_p[wave], s_alpha[wave], is_res, nvalid, a.qk_scale, a.beta_log2,
                           col, grp, c, ph, vc, s0);
  }
  // wave state -> LDS: sum the row phases of acc, keep max and sum per head
#pragma unroll
  for (int msk = Regs::CPR; msk < 64; msk <<= 1)
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) st.acc[h][e] = wave_xor_add(st.acc[h][e], msk);
  if (ph == 0) {
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) s_acc[wave][h][8 * c + e] = st.acc[h][e];
  }
  if (col == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * grp + i;
      if (h < GP) {
        s_m[wave][h] = st.m[i];
        s_l[wave][h] = st.l[i];
      }
    }
  }
  __syncthreads();
  // merge the 4 waves into this block's record
  const size_t rec = ((size_t)bh * a.P + p) * GP;
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
    a.part_acc[(rec + h) * D + d] = o;
    if (d == 0) {
      a.part_ml[(rec + h) * 2 + 0] = M;
      a.part_ml[(rec + h) * 2 + 1] = l;
    }
  }
}

// Merge the records of one (b, kv head), evaluate the gate and write the G
// outputs. Record p < PR is residual chunk p, record PR + q is main chunk q;
// only chunks that hold slots were written.
template <int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_combine(DecodeArgs a) {
  extern __shared__ float s_w[];  // [GP][P] weights of the records
  const int kvh = blockIdx.x, b = blockIdx.y;
  const int bh = b * a.Hkv + kvh;
  int r, n;
  cache_lengths(a.res_len, a.main_len, bh, a.C, a.Rcap, r, n);
  const int nRC = (r + kChunk - 1) / kChunk, nMC = (n + kChunk - 1) / kChunk;
  const float* ml = a.part_ml + (size_t)bh * a.P * GP * 2;
  const float* pacc = a.part_acc + (size_t)bh * a.P * GP * D;
  const int tid = threadIdx.x, lane16 = tid & 15, h = tid >> 4;
  if (h < a.G) {
    float mM = kNegInf, mR = kNegInf;
    for (int q = lane16; q < nMC; q += 16) mM = fmaxf(mM, ml[((a.PR + q) * GP + h) * 2]);
    for (int q = lane16; q < nRC; q += 16) mR = fmaxf(mR, ml[(q * GP + h) * 2]);
#pragma unroll
    for (int msk = 1; msk < 16; msk <<= 1) { mM = wave_xor_max(mM, msk); mR = wave_xor_max(mR, msk); }
    float lM = 0.f, lR = 0.f;
    for (int q = lane16; q < nMC; q += 16) {
      const float* e = ml + ((a.PR + q) * GP + h) * 2;
      if (e[0] != kNegInf) lM = fmaf(e[1], exp2f(e[0] - mM), lM);
    }
    for (int q = lane16; q < nRC; q += 16) {
      const float* e = ml + (q * GP + h) * 2;
      if (e[0] != kNegInf) lR = fmaf(e[1], exp2f(e[0] - mR), lR);
    }
#pragma unroll
    for (int msk = 1; msk < 16; msk <<= 1) { lM = wave_xor_add(lM, msk); lR = wave_xor_add(lR, msk); }
    // p_max = max_p e^{a_p} / sum_p e^{a_p} = 1 / lM: the max term is exactly 1
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
    const float inv = den > 0.f ? 1.f / den : 0.f;
    for (int q = lane16; q < nMC; q += 16) {
      const float m = ml[((a.PR + q) * GP + h) * 2];
      s_w[h * a.P + a.PR + q] = m != kNegInf ? exp2f(m - Mx) * inv : 0.f;
    }
    for (int q = lane16; q < nRC; q += 16) {
      const float m = ml[(q * GP + h) * 2];
      s_w[h * a.P + q] = (m != kNegInf && mRg != kNegInf) ? exp2f(m + lg2g - Mx) * inv : 0.f;
    }
    if (lane16 == 0) {
      if (a.dbg_lse_main) a.dbg_lse_main[qh] = lM > 0.f ? (mM + log2f(lM)) * kLn2 : kNegInf;
      if (a.dbg_lse_res) a.dbg_lse_res[qh] = lR > 0.f ? (mR + log2f(lR)) * kLn2 : kNegInf;
      if (a.dbg_gate) a.dbg_gate[qh] = g;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < a.G * D; idx += kThreads) {
    const int hh = idx / D, d = idx % D;
    const float* w = s_w + hh * a.P;
    float o0 = 0.f, o1 = 0.f;
    int q = 0;
    for (; q + 1 < nRC; q += 2) {
      o0 = fmaf(w[q], pacc[(q * GP + hh) * D + d], o0);
      o1 = fmaf(w[q + 1], pacc[((q + 1) * GP + hh) * D + d], o1);
    }
    if (q < nRC) o0 = fmaf(w[q], pacc[(q * GP + hh) * D + d], o0);
    for (q = 0; q + 1 < nMC; q += 2) {
      const int pp = a.PR + q;
      o0 = fmaf(w[pp], pacc[(pp * GP + hh) * D + d], o0);
      o1 = fmaf(w[pp + 1], pacc[((pp + 1) * GP + hh) * D + d], o1);
    }
    if (q < nMC) o0 = fmaf(w[a.PR + q], pacc[((a.PR + q) * GP + hh) * D + d], o0);
    a.out[((size_t)b * a.Hq + kvh * a.G + hh) * D + d] = o0 + o1;
  }
}


// One block of 16 waves per (b, kv head): streams every slot of the head,
// merges the wave states in LDS, applies the gate and writes the G outputs;
// optionally appends this step's token first. Used when the (b, kv head)
// pairs alone fill the GPU, so no split-K records or second launch are needed.
// 8 waves (2 per SIMD, up to 256 registers each): every variant that needed
// more registers (a second key buffer for prefetch, or 12-16 waves) spilled
// to scratch and ran 1.5-3x slower.
constexpr int kHeadWaves = 8;
constexpr int kHeadThreads = 64 * kHeadWaves;

template <typename T, int D, int GP>
__global__ __launch_bounds__(kHeadThreads) void decode_head(DecodeArgs a) {
  using Regs = VRegs<T, D>;
  const int kvh = blockIdx.x, b = blockIdx.y;
  const int bh = b * a.Hkv + kvh;
  int r, n;
  cache_lengths(a.res_len, a.main_len, bh, a.C, a.Rcap, r, n);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int c = lane % Regs::CPR, ph = lane / Regs::CPR;
  T* kc = static_cast<T*>(const_cast<void*>(a.kc)) + (size_t)bh * a.C * D;
  T* vc = static_cast<T*>(const_cast<void*>(a.vc)) + (size_t)bh * a.C * D;
  const float* logc = a.logc + (size_t)bh * a.Rcap;

  // fused append of this step's token as main slot r + n (Sec. 3.1)
  const bool app = a.k_new != nullptr && r + n < a.C;
  if (app) {
    const T* kn = static_cast<const T*>(a.k_new) + (size_t)bh * D;
    const T* vn = static_cast<const T*>(a.v_new) + (size_t)bh * D;
    for (int x = tid; x < D; x += kHeadThreads) {
      kc[(size_t)(r + n) * D + x] = kn[x];
      vc[(size_t)(r + n) * D + x] = vn[x];
    }
  }
  __syncthreads();  // the appended row is visible to every wave of the block
  if (app) n += 1;

  __shared__ float s_p[kHeadWaves][kUnit][GP];
  __shared__ float s_alpha[kHeadWaves][GP];
  __shared__ float s_acc[kHeadWaves][GP][D];
  __shared__ float s_m[kHeadWaves][GP];
  __shared__ float s_l[kHeadWaves][GP];
  __shared__ float s_res[GP][D + 2];  // merged residual state: acc[D], m, l

  QK<T, D> qk;
  qk.load_q(static_cast<const T*>(a.q) + ((size_t)b * a.Hq + (size_t)kvh * a.G + col) * D + grp * (D / 4),
            col < a.G);

  for (int kind = 0; kind < 2; ++kind) {
    const bool is_res = kind == 0;
    const int base = is_res ? 0 : r;
    const int end = is_res ? r : r + n;
    const int U = (end - base + kUnit - 1) / kUnit;
    WaveState<GP> st;
    st.reset();
    for (int u = wave; u < U; u += kHeadWaves) {  // wave-uniform
      const int s0 = base + u * kUnit;
      const int nvalid = min(kUnit, end - s0);
      KRegs<T, D> kr;
      VRegs<T, D> vr;
      load_unit_k<T, D>(kr, kc, logc, is_res, s0, nvalid, col, grp);
      process_unit<T, D, GP>(kr, vr, qk, st, s_p[wave], s_alpha[wave], is_res, nvalid, a.qk_scale, a.beta_log2,
                             col, grp, c, ph, vc, s0);
    }
#pragma unroll
    for (int msk = Regs::CPR; msk < 64; msk <<= 1)
#pragma unroll
      for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) st.acc[h][e] = wave_xor_add(st.acc[h][e], msk);
    if (ph == 0) {
#pragma unroll
      for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) s_acc[wave][h][8 * c + e] = st.acc[h][e];
    }
    if (col == 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int h = 4 * grp + i;
        if (h < GP) {
          s_m[wave][h] = st.m[i];
          s_l[wave][h] = st.l[i];
        }
      }
    }
    __syncthreads();
    for (int idx = tid; idx < GP * D; idx += kHeadThreads) {
      const int h = idx / D, d = idx % D;
      float M = s_m[0][h];
#pragma unroll
      for (int w = 1; w < kHeadWaves; ++w) M = fmaxf(M, s_m[w][h]);
      float o = 0.f, l = 0.f;
      if (M != kNegInf) {
#pragma unroll
        for (int w = 0; w < kHeadWaves; ++w) {
          const float f = exp2f(s_m[w][h] - M);
          o = fmaf(f, s_acc[w][h][d], o);
          l = fmaf(f, s_l[w][h], l);
        }
      }
      if (is_res) {
        s_res[h][d] = o;
        if (d == 0) { s_res[h][D] = M; s_res[h][D + 1] = l; }
        continue;
      }
      if (h >= a.G) continue;
      // main merged: p_max = 1 / l (the max term is exactly 1), then the gate
      const float pmax = l > 0.f ? 1.f / l : 1.f;
      const int qh = b * a.Hq + kvh * a.G + h;
      const float tau = a.tau ? a.tau[qh] : a.tau_scalar;
      const float g = fmaxf(a.g_min, 1.f / (1.f + expf(-(tau - pmax) * a.alpha)));
      const float lg2g = g > 0.f ? log2f(g) : kNegInf;
      const float mR = s_res[h][D], lR = s_res[h][D + 1];
      const float mRg = (mR == kNegInf || lg2g == kNegInf) ? kNegInf : mR + lg2g;
      const float Mx = fmaxf(M, mRg);
      const float fM = M != kNegInf ? exp2f(M - Mx) : 0.f;
      const float fR = mRg != kNegInf ? exp2f(mRg - Mx) : 0.f;
      const float den = l * fM + lR * fR;
      const float num = o * fM + s_res[h][d] * fR;
      a.out[(size_t)qh * D + d] = den > 0.f ? num / den : 0.f;
      if (d == 0) {
        if (a.dbg_lse_main) a.dbg_lse_main[qh] = l > 0.f ? (M + log2f(l)) * kLn2 : kNegInf;
        if (a.dbg_lse_res) a.dbg_lse_res[qh] = lR > 0.f ? (mR + log2f(lR)) * kLn2 : kNegInf;
        if (a.dbg_gate) a.dbg_gate[qh] = g;
      }
    }
    __syncthreads();
  }
  if (app && tid == 0) a.main_len[bh] = n;
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
hipError_t launch_typed(const DecodePlan& pl, const DecodeArgs& da, hipStream_t stream) {
  if constexpr (GP <= 4) {
    if (pl.whole_head) {
      hipLaunchKernelGGL((decode_head<T, D, GP>), dim3(pl.Hkv, pl.B), dim3(kHeadThreads), 0, stream, da);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((decode_split<T, D, GP>), dim3(pl.P, pl.Hkv, pl.B), dim3(kThreads), 0, stream, da);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = (size_t)GP * pl.P * sizeof(float);
  hipLaunchKernelGGL((decode_combine<D, GP>), dim3(pl.Hkv, pl.B), dim3(kThreads), lds, stream, da);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_gp(const DecodePlan& pl, const DecodeArgs& da, hipStream_t stream) {
  switch (pl.GP) {
    case 1: return launch_typed<T, D, 1>(pl, da, stream);
    case 2: return launch_typed<T, D, 2>(pl, da, stream);
    case 4: return launch_typed<T, D, 4>(pl, da, stream);
    case 8: return launch_typed<T, D, 8>(pl, da, stream);
    case 16: return launch_typed<T, D, 16>(pl, da, stream);
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
  p.PR = (rmax + kChunk - 1) / kChunk;
  p.P = p.PR + (s.slot_cap + kChunk - 1) / kChunk;
  // one block per (b, kv head) when those alone fill the chip's CUs
  p.whole_head = p.GP <= 4 && (long long)p.B * p.Hkv >= kWholeHeadMin;
  const size_t recs = (size_t)p.B * p.Hkv * p.P * p.GP;
  p.acc_off = 0;
  p.ml_off = align_up(recs * p.D * sizeof(float), 256);
  p.bytes = p.ml_off + align_up(recs * 2 * sizeof(float), 256);
  return p;
}

size_t decode_max_lds_weights() { return 48 * 1024; }

hipError_t launch_decode(const reskv_shape_t& s, const reskv_gate_t& g, const DecodePlan& pl,
                         const void* q, void* kc, void* vc, const float* logc,
                         const int32_t* res_len, int32_t* main_len, const void* k_new, const void* v_new,
                         float* out, float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate,
                         void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  if (k_new && !pl.whole_head) {  // split-K path: append as its own launch first
    const hipError_t e = launch_append(s, k_new, v_new, kc, vc, res_len, main_len, stream);
    if (e != hipSuccess) return e;
  }
  DecodeArgs da{};
  if (pl.whole_head) { da.k_new = k_new; da.v_new = v_new; }
  da.q = q; da.kc = kc; da.vc = vc; da.logc = logc;
  da.res_len = res_len; da.main_len = main_len;
  da.part_acc = reinterpret_cast<float*>(ws + pl.acc_off);
  da.part_ml = reinterpret_cast<float*>(ws + pl.ml_off);
  da.tau = g.tau; da.out = out;
  da.dbg_lse_main = dbg_lse_main; da.dbg_lse_res = dbg_lse_res; da.dbg_gate = dbg_gate;
  da.Hq = pl.Hq; da.Hkv = pl.Hkv; da.G = pl.G; da.C = pl.C; da.Rcap = pl.Rcap; da.PR = pl.PR; da.P = pl.P;
  da.qk_scale = kLog2e / sqrtf((float)pl.D);
  da.beta_log2 = g.beta * kLog2e;
  da.tau_scalar = g.tau_scalar; da.alpha = g.alpha; da.g_min = g.g_min;
  const bool bf = s.dtype == RESKV_BF16;
  if (pl.D == 128) return bf ? launch_gp<uint16_t, 128>(pl, da, stream) : launch_gp<float, 128>(pl, da, stream);
  if (pl.D == 64) return bf ? launch_gp<uint16_t, 64>(pl, da, stream) : launch_gp<float, 64>(pl, da, stream);
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
