// Shared-softmax residual decode (Sec. 5.4; Sec. 5.5.2 gate; App. D, Algorithm 2).
//
// Flash decode over the fixed-budget cache of one layer. Two shapes:
//   decode_head    one block of 8 waves per (b, kv head) streams every slot
//                  of the head, merges the waves in LDS, applies the gate
//                  and writes the outputs (used when the (b, kv head) pairs
//                  alone fill the GPU); it can append this step's token.
//   decode_split + decode_combine
//                  split-K: one block = 256 slots of one (b, kv head), all of
//                  one kind (residual slots [0, r) or main slots [r, r+n)),
//                  writes a partial record (max m, sum l, unnormalised acc)
//                  per query head; the combine merges the main records
//                  (p_max = 1 / l_main: the max term contributes exactly 1),
//                  evaluates the gate, shifts the residual records by log g
//                  and gives main and residual one shared denominator.
// The combine is a separate launch rather than a last-arriving-block epilogue:
// on this multi-XCD part a device-scope release/acquire per block writes back
// and invalidates L2, which costs far more than one more launch.
//
// One wave handles a unit of 64 slots entirely in registers. With
// hd = lane % 16 and g = lane / 16:
//   * logits S^T = K Q^T on MFMA per 16-slot tile t (A = key rows, B = query
//     rows), so lane (hd, g) holds S[slot 16t + 4g + i][head hd], i = 0..3;
//     logits are kept in base 2 with log2(e)/sqrt(d) folded into one scale;
//   * the per-head max and sum run over the lane's 16 values, then across
//     the four lane groups;
//   * O^T += V^T P^T on MFMA: lane (m, g) loads the m-th (D/16)-element piece
//     of value rows 16T + 4g + u, which is exactly the A operand when the
//     MFMA contraction index k = 8g + i' stands for slot
//     16(2h + i'/4) + 4g + i'%4 (k-step h); the B operand is then the lane's
//     own probabilities. bf16 probabilities are split into hi + lo bf16 parts
//     (two MFMAs), fp32 caches use the fp32 MFMA. Lane (hd, g) ends with
//     O[head hd][columns g*D/4 .. (g+1)*D/4), so rescaling by the per-head
//     alpha and the final write need no cross-lane traffic.
#include <mutex>

#include "common.h"
#include "internal.h"

namespace reskv {

// Scratch of the allocation-free decode entry point: split-K records live in
// this file-scope device array instead of a caller workspace. Each GPU the
// library runs on holds its own copy until the process ends; host code uses
// the device address hipGetSymbolAddress returns for the current device,
// never the array's name.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kUnit = 64;              // slots per wave unit
constexpr int kTiles = kUnit / 16;     // 16-slot MFMA tiles per unit
constexpr int kChunk = kWaves * kUnit; // slots per split block
constexpr int kWholeHeadMin = 256;     // (b, kv head) pairs that fill the 256 CUs

struct DecodeArgs {
  const void* q;
  const void* kc;
  const void* vc;
  const float* logc;
  const int32_t* res_len;
  int32_t* main_len;
  const void* k_new;  // fused append of this step's token, or NULL
  const void* v_new;
  float* part_acc;  // [B*Hkv][P][GP][D]
  float* part_ml;   // [B*Hkv][P][GP][2]  (m in base 2, l)
  const float* tau;
  float* out;
  float* dbg_lse_main;
  float* dbg_lse_res;
  float* dbg_gate;
  float* out_res;   // two-branch mode: the residual branch's own output (out = the main branch's)
  int32_t* plan;    // ragged schedule: [BH] unit prefix, then U and the block count
  float* rec;       // ragged schedule: [blocks][2 edges][2 kinds][GP][D + 2] partial states
  int Hq, Hkv, G, C, Rcap, PR, P;
  int BH;           // B * Hkv
  int rag_blocks;   // ragged schedule: at least this many blocks (one per CU)
  int rag_min_units;  // ragged schedule: at least this many units per block
  float qk_scale;   // log2(e) / sqrt(d)
  float beta_log2;  // beta * log2(e)
  float tau_scalar, alpha, g_min;
};

__device__ __forceinline__ void cache_lengths(const int32_t* res_len, const int32_t* main_len,
                                              int bh, int C, int Rcap, int& r, int& n) {
  r = clampi(res_len[bh], 0, min(Rcap, C));
  n = clampi(main_len[bh], 0, C - r);
}

// Raw words of one value-row piece (D/16 elements) of one lane.
template <typename T, int D>
struct VPiece {
  static constexpr int kElems = D / 16;
  static constexpr int kWords = kElems * (int)sizeof(T) / 4;
  uint32_t w[kWords];
  __device__ __forceinline__ void load(const T* p) {
    if constexpr (kWords == 2) {
      const uint2 x = *reinterpret_cast<const uint2*>(p);
      w[0] = x.x; w[1] = x.y;
    } else {
#pragma unroll
      for (int j = 0; j < kWords / 4; ++j) {
        const uint4 x = reinterpret_cast<const uint4*>(p)[j];
        w[4 * j] = x.x; w[4 * j + 1] = x.y; w[4 * j + 2] = x.z; w[4 * j + 3] = x.w;
      }
    }
  }
  __device__ __forceinline__ void store(T* p) const {
    if constexpr (kWords == 2) {
      *reinterpret_cast<uint2*>(p) = make_uint2(w[0], w[1]);
    } else {
#pragma unroll
      for (int j = 0; j < kWords / 4; ++j)
        reinterpret_cast<uint4*>(p)[j] = make_uint4(w[4 * j], w[4 * j + 1], w[4 * j + 2], w[4 * j + 3]);
    }
  }
};

// Key fragments (+ log-counts) and value pieces of one 64-slot unit.
template <typename T, int D>
struct UnitRegs {
  Frag<T, D> k[kTiles];    // key row 16t + hd
  float lc[kTiles][4];     // log-count of slot 16t + 4g + i (residual units)
  VPiece<T, D> v[16];      // v[4T + u]: piece hd of value row 16T + 4g + u
};

// Key rows s0 + 16t + hd of a unit, clamped to row `last` (rows past the
// valid range get no probability). Slot app_row (or none if -1) is taken from
// the token being appended (kn) instead of the cache; only the unit that
// holds it (a wave-uniform test) pays for the per-lane pointer choice.
template <typename T, int D>
__device__ __forceinline__ void load_unit_k(UnitRegs<T, D>& u, const T* kc, int s0, int last, int hd, int g,
                                            int app_row, const T* kn) {
  if (app_row >= s0 && app_row < s0 + kUnit) {
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
      const int row = min(s0 + 16 * t + hd, last);
      u.k[t].load(row == app_row ? kn : kc + (size_t)row * D, g);
    }
  } else {
#pragma unroll
    for (int t = 0; t < kTiles; ++t) u.k[t].load(kc + (size_t)min(s0 + 16 * t + hd, last) * D, g);
  }
}

// Log-counts of the unit's residual slots s0 + j, j < nres.
template <typename T, int D>
__device__ __forceinline__ void load_unit_lc(UnitRegs<T, D>& u, const float* logc, int s0, int nres, int g) {
#pragma unroll
  for (int t = 0; t < kTiles; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 16 * t + 4 * g + i;
      u.lc[t][i] = j < nres ? logc[s0 + j] : 0.f;
    }
}

// Value rows of unit [s0, s0 + nvalid), clamped into the unit; slot app_row
// from vn as for the keys.
template <typename T, int D>
__device__ __forceinline__ void load_unit_v(UnitRegs<T, D>& u, const T* vc, int s0, int nvalid, int hd, int g,
                                            int app_row, const T* vn) {
  constexpr int kE = VPiece<T, D>::kElems;
  if (app_row >= s0 && app_row < s0 + nvalid) {
#pragma unroll
    for (int T4 = 0; T4 < 4; ++T4)
#pragma unroll
      for (int uu = 0; uu < 4; ++uu) {
        const int row = s0 + min(16 * T4 + 4 * g + uu, nvalid - 1);
        u.v[4 * T4 + uu].load((row == app_row ? vn : vc + (size_t)row * D) + kE * hd);
      }
  } else {
#pragma unroll
    for (int T4 = 0; T4 < 4; ++T4)
#pragma unroll
      for (int uu = 0; uu < 4; ++uu)
        u.v[4 * T4 + uu].load(vc + (size_t)(s0 + min(16 * T4 + 4 * g + uu, nvalid - 1)) * D + kE * hd);
  }
}

// Online-softmax state of one wave for one kind: head hd's running max and
// sum (replicated over the four lane groups) and O^T tiles (lane (hd, g)
// holds O[hd][(D/16)(4g + i) + e] in acc[e][i]).
template <int D>
struct WaveState {
  static constexpr int kE = D / 16;
  float m, l;
  f32x4_t acc[kE];
  __device__ void reset() {
    m = kNegInf;
    l = 0.f;
#pragma unroll
    for (int e = 0; e < kE; ++e) acc[e] = zero4();
  }
};

// bf16 halves of two fp32 values packed into one word (a low, b high),
// truncating; perm selector 0x07060302 takes the upper halves of both.
__device__ __forceinline__ uint32_t pack_hi(float a, float b) {
  return __builtin_amdgcn_perm(__float_as_uint(b), __float_as_uint(a), 0x07060302u);
}
__device__ __forceinline__ float trunc_bf16(float x) { return __uint_as_float(__float_as_uint(x) & 0xffff0000u); }

// P.V of one unit: O^T tiles += V^T P^T (see the file comment for the
// slot order of the contraction index).
template <int D>
__device__ __forceinline__ void pv_unit(WaveState<D>& st, const UnitRegs<uint16_t, D>& u, const float (&p)[kTiles][4]) {
  constexpr int kE = D / 16;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    // B operands: probabilities of slots 16(2h + i'/4) + 4g + i'%4, i' = 0..7,
    // as bf16 hi and lo parts
    uint32_t bh[4], bl[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float pa = p[2 * h + (2 * w) / 4][(2 * w) % 4];
      const float pb = p[2 * h + (2 * w + 1) / 4][(2 * w + 1) % 4];
      bh[w] = pack_hi(pa, pb);
      bl[w] = pack_hi(pa - trunc_bf16(pa), pb - trunc_bf16(pb));
    }
    const bf16x8_t Bh = __builtin_bit_cast(bf16x8_t, make_uint4(bh[0], bh[1], bh[2], bh[3]));
    const bf16x8_t Bl = __builtin_bit_cast(bf16x8_t, make_uint4(bl[0], bl[1], bl[2], bl[3]));
#pragma unroll
    for (int e = 0; e < kE; ++e) {
      // A operand: element e of value rows 8h + i', packed in pairs
      const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
      uint32_t av[4];
#pragma unroll
      for (int w = 0; w < 4; ++w)
        av[w] = __builtin_amdgcn_perm(u.v[8 * h + 2 * w + 1].w[e >> 1], u.v[8 * h + 2 * w].w[e >> 1], sel);
      const bf16x8_t A = __builtin_bit_cast(bf16x8_t, make_uint4(av[0], av[1], av[2], av[3]));
      st.acc[e] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, Bh, st.acc[e], 0, 0, 0);
      st.acc[e] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, Bl, st.acc[e], 0, 0, 0);
    }
  }
}

template <int D>
__device__ __forceinline__ void pv_unit(WaveState<D>& st, const UnitRegs<float, D>& u, const float (&p)[kTiles][4]) {
  constexpr int kE = D / 16;
#pragma unroll
  for (int T4 = 0; T4 < 4; ++T4)
#pragma unroll
    for (int uu = 0; uu < 4; ++uu)
#pragma unroll
      for (int e = 0; e < kE; ++e)
        st.acc[e] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(u.v[4 * T4 + uu].w[e]), p[T4][uu],
                                                         st.acc[e], 0, 0, 0);
}

// Scaled logits of one unit in base 2: lane (hd, g) gets slot 16t + 4g + i.
template <typename T, int D>
__device__ __forceinline__ void unit_logits(const UnitRegs<T, D>& u, const Frag<T, D>& q, float qk_scale,
                                            float (&s)[kTiles][4]) {
#pragma unroll
  for (int t = 0; t < kTiles; ++t) {
    const f32x4_t c = mma<D>(u.k[t], q, zero4());
#pragma unroll
    for (int i = 0; i < 4; ++i) s[t][i] = c[i] * qk_scale;
  }
}

// Online softmax update over the unit's slots [lo, hi) of one kind (residual
// slots add beta * log2 count; empty entries and other slots get no weight):
// per-head max and sum over the lane's 16 slots, then across the four lane
// groups, then P.V.
template <typename T, int D>
__device__ __forceinline__ void softmax_pv(WaveState<D>& st, const UnitRegs<T, D>& u, const float (&s)[kTiles][4],
                                           int lo, int hi, bool is_res, float beta_log2, int g) {
  float p[kTiles][4];
  float mloc = kNegInf;
#pragma unroll
  for (int t = 0; t < kTiles; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 16 * t + 4 * g + i;
      const bool live = j >= lo && j < hi && !(is_res && u.lc[t][i] == kNegInf);
      const float v = is_res ? fmaf(beta_log2, u.lc[t][i], s[t][i]) : s[t][i];
      p[t][i] = live ? v : kNegInf;
      mloc = fmaxf(mloc, p[t][i]);
    }
  mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
  mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
  const float m_new = fmaxf(st.m, mloc);
  const float mu = (m_new == kNegInf) ? 0.f : m_new;
  const float alpha = fast_exp2(st.m - mu);
  float lsum = 0.f;
#pragma unroll
  for (int t = 0; t < kTiles; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[t][i] = fast_exp2(p[t][i] - mu);
      lsum += p[t][i];
    }
  lsum += __shfl_xor(lsum, 16, 64);
  lsum += __shfl_xor(lsum, 32, 64);
  st.l = fmaf(st.l, alpha, lsum);
  st.m = m_new;
#pragma unroll
  for (int e = 0; e < WaveState<D>::kE; ++e)
#pragma unroll
    for (int i = 0; i < 4; ++i) st.acc[e][i] *= alpha;
  pv_unit<D>(st, u, p);
}

// Wave state -> LDS rows of the query heads this block serves: acc as
// [GP][D], max and sum per head.
template <int D, int GP>
__device__ __forceinline__ void store_wave_state(const WaveState<D>& st, float (*acc)[D], float* m, float* l,
                                                 int hd, int g) {
  if (hd < GP) {
    constexpr int kE = D / 16;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < kE; ++e) acc[hd][kE * (4 * g + i) + e] = st.acc[e][i];
    if (g == 0) {
      m[hd] = st.m;
      l[hd] = st.l;
    }
  }
}

template <typename T, int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_split(DecodeArgs a) {
  const int p = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  int r, n;
  cache_lengths(a.res_len, a.main_len, bh, a.C, a.Rcap, r, n);
  // fused append: this step's token is main slot r + n, read from k_new /
  // v_new and stored into the cache by the wave whose unit holds it;
  // decode_combine advances main_len once every block has read it
  const bool app = a.k_new != nullptr && r + n < a.C;
  const int app_row = app ? r + n : -1;
  const T* kn = app ? static_cast<const T*>(a.k_new) + (size_t)bh * D : nullptr;
  const T* vn = app ? static_cast<const T*>(a.v_new) + (size_t)bh * D : nullptr;
  if (app) n += 1;
  // block p < PR covers residual slots [256p, 256p + 256) of [0, r); block
  // p >= PR covers main slots [r + 256(p-PR), ...) of [r, r + n)
  const bool is_res = p < a.PR;
  const int base = is_res ? 0 : r;
  const int end = is_res ? r : r + n;
  const int lo = base + (is_res ? p : p - a.PR) * kChunk;
  if (lo >= end) return;  // block-uniform

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hd = lane & 15, g = lane >> 4;

  __shared__ float s_acc[kWaves][GP][D];
  __shared__ float s_m[kWaves][GP];
  __shared__ float s_l[kWaves][GP];

  const T* kc = static_cast<const T*>(a.kc) + (size_t)bh * a.C * D;
  const T* vc = static_cast<const T*>(a.vc) + (size_t)bh * a.C * D;
  const float* logc = a.logc + (size_t)bh * a.Rcap;

  WaveState<D> st;
  st.reset();
  const int s0 = lo + wave * kUnit;
  if (s0 < end) {  // wave-uniform
    Frag<T, D> q;
    if (hd < a.G) q.load(static_cast<const T*>(a.q) + ((size_t)b * a.Hq + (size_t)kvh * a.G + hd) * D, g);
    else q.zero();
    UnitRegs<T, D> u;
    const int nvalid = min(kUnit, end - s0);
    load_unit_k<T, D>(u, kc, s0, end - 1, hd, g, app_row, kn);
    if (is_res) load_unit_lc<T, D>(u, logc, s0, nvalid, g);
    // the value rows are requested before the logits wait on the keys
    load_unit_v<T, D>(u, vc, s0, nvalid, hd, g, app_row, vn);
    float sc[kTiles][4];
    unit_logits<T, D>(u, q, a.qk_scale, sc);
    softmax_pv<T, D>(st, u, sc, 0, nvalid, is_res, a.beta_log2, g);
    if (app_row >= s0 && app_row < s0 + nvalid) {  // wave-uniform: the new rows into the cache
      constexpr int kPieces = D * (int)sizeof(T) / 16;
      if (lane < 2 * kPieces) {
        const bool isv = lane >= kPieces;
        const int c = isv ? lane - kPieces : lane;
        T* dst = static_cast<T*>(const_cast<void*>(isv ? a.vc : a.kc)) + ((size_t)bh * a.C + app_row) * D;
        reinterpret_cast<uint4*>(dst)[c] = reinterpret_cast<const uint4*>(isv ? vn : kn)[c];
      }
    }
  }
  store_wave_state<D, GP>(st, s_acc[wave], s_m[wave], s_l[wave], hd, g);
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
// only chunks that hold slots were written. The loads that do not depend on
// the cache lengths are issued before those arrive: the (max, sum) of the
// first 16 kML records of this thread's query head and the accumulators of
// the first kPF records of its outputs. Records of chunks without slots hold
// stale values; they are masked once the lengths are known.
template <int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_combine(DecodeArgs a) {
  extern __shared__ float s_w[];  // [GP][P] weights of the records
  const int kvh = blockIdx.x, b = blockIdx.y;
  const int bh = b * a.Hkv + kvh;
  const int tid = threadIdx.x, lane16 = tid & 15, h = tid >> 4;
  const float2* ml = reinterpret_cast<const float2*>(a.part_ml) + (size_t)bh * a.P * GP;
  const float* pacc = a.part_acc + (size_t)bh * a.P * GP * D;
  constexpr int kML = 4;
  constexpr int kOut = (GP * D + kThreads - 1) / kThreads;
  constexpr int kPF = kOut >= 8 ? 8 : 16;
  const bool hv = h < a.G;
  float2 mlv[kML];
#pragma unroll
  for (int k = 0; k < kML; ++k) {
    const int q = lane16 + 16 * k;
    mlv[k] = hv && q < a.P ? ml[q * GP + h] : make_float2(kNegInf, 0.f);
  }
  float pv[kOut][kPF];
#pragma unroll
  for (int k = 0; k < kOut; ++k) {
    const int idx = min(tid + k * kThreads, a.G * D - 1), hh = idx / D, d = idx % D;
#pragma unroll
    for (int j = 0; j < kPF; ++j) pv[k][j] = j < a.P ? pacc[(j * GP + hh) * D + d] : 0.f;
  }
  int r, n;
  cache_lengths(a.res_len, a.main_len, bh, a.C, a.Rcap, r, n);
  const bool app = a.k_new != nullptr && r + n < a.C;  // as in decode_split
  if (app) n += 1;
  const int nRC = (r + kChunk - 1) / kChunk, nMC = (n + kChunk - 1) / kChunk;
  auto valid = [&](int p) { return p < nRC || (p >= a.PR && p < a.PR + nMC); };
  if (hv) {
    auto rec = [&](int k, int p) { return k < kML ? mlv[k] : ml[p * GP + h]; };
    float mM = kNegInf, mR = kNegInf;
    for (int k = 0, p = lane16; p < a.P; ++k, p += 16) {
      if (!valid(p)) continue;
      const float m = rec(k, p).x;
      if (p >= a.PR) mM = fmaxf(mM, m);
      else mR = fmaxf(mR, m);
    }
#pragma unroll
    for (int msk = 1; msk < 16; msk <<= 1) { mM = wave_xor_max(mM, msk); mR = wave_xor_max(mR, msk); }
    float lM = 0.f, lR = 0.f;
    for (int k = 0, p = lane16; p < a.P; ++k, p += 16) {
      const float2 e = rec(k, p);
      if (!valid(p) || e.x == kNegInf) continue;
      if (p >= a.PR) lM = fmaf(e.y, exp2f(e.x - mM), lM);
      else lR = fmaf(e.y, exp2f(e.x - mR), lR);
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
    for (int k = 0, p = lane16; p < a.P; ++k, p += 16) {
      const float m = rec(k, p).x;
      float w = 0.f;
      if (valid(p) && m != kNegInf) {
        if (p >= a.PR) w = exp2f(m - Mx) * inv;
        else if (mRg != kNegInf) w = exp2f(m + lg2g - Mx) * inv;
      }
      s_w[h * a.P + p] = w;
    }
    if (lane16 == 0) {
      if (a.dbg_lse_main) a.dbg_lse_main[qh] = lM > 0.f ? (mM + log2f(lM)) * kLn2 : kNegInf;
      if (a.dbg_lse_res) a.dbg_lse_res[qh] = lR > 0.f ? (mR + log2f(lR)) * kLn2 : kNegInf;
      if (a.dbg_gate) a.dbg_gate[qh] = g;
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kOut; ++k) {
    const int idx = tid + k * kThreads;
    if (idx >= a.G * D) continue;
    const int hh = idx / D, d = idx % D;
    const float* w = s_w + hh * a.P;
    float o = 0.f;
#pragma unroll
    for (int j = 0; j < kPF; ++j)
      if (j < a.P && valid(j)) o = fmaf(w[j], pv[k][j], o);
    for (int j = kPF; j < a.P; ++j)
      if (valid(j)) o = fmaf(w[j], pacc[(j * GP + hh) * D + d], o);
    a.out[((size_t)b * a.Hq + kvh * a.G + hh) * D + d] = o;
  }
  // the appended token is in the cache: advance main_len (one block per
  // head, and every thread of it read the length above)
  if (app && tid == 0) a.main_len[bh] = n;
}


// Two-branch combine: the split records of each kind are merged under that
// kind's own softmax. out = main-branch output, out_res = residual-branch
// output (0 without populated entries), dbg_lse_main / dbg_lse_res their
// natural log-sum-exp (the residual one without the gate), dbg_gate the gate.
template <int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_branches(DecodeArgs a) {
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
    const float pmax = lM > 0.f ? 1.f / lM : 1.f;
    const int qh = b * a.Hq + kvh * a.G + h;
    const float tau = a.tau ? a.tau[qh] : a.tau_scalar;
    const float g = fmaxf(a.g_min, 1.f / (1.f + expf(-(tau - pmax) * a.alpha)));
    const float invM = lM > 0.f ? 1.f / lM : 0.f, invR = lR > 0.f ? 1.f / lR : 0.f;
    for (int q = lane16; q < nMC; q += 16) {
      const float m = ml[((a.PR + q) * GP + h) * 2];
      s_w[h * a.P + a.PR + q] = m != kNegInf ? exp2f(m - mM) * invM : 0.f;
    }
    for (int q = lane16; q < nRC; q += 16) {
      const float m = ml[(q * GP + h) * 2];
      s_w[h * a.P + q] = m != kNegInf ? exp2f(m - mR) * invR : 0.f;
    }
    if (lane16 == 0) {
      a.dbg_lse_main[qh] = lM > 0.f ? (mM + log2f(lM)) * kLn2 : kNegInf;
      a.dbg_lse_res[qh] = lR > 0.f ? (mR + log2f(lR)) * kLn2 : kNegInf;
      a.dbg_gate[qh] = g;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < a.G * D; idx += kThreads) {
    const int hh = idx / D, d = idx % D;
    const float* w = s_w + hh * a.P;
    float oR = 0.f, oM = 0.f;
    for (int q = 0; q < nRC; ++q) oR = fmaf(w[q], pacc[(q * GP + hh) * D + d], oR);
    for (int q = 0; q < nMC; ++q) oM = fmaf(w[a.PR + q], pacc[((a.PR + q) * GP + hh) * D + d], oM);
    const size_t o = ((size_t)b * a.Hq + kvh * a.G + hh) * D + d;
    a.out[o] = oM;
    a.out_res[o] = oR;
  }
}

// Merge of the two branches, one thread per output element: the
// log-sum-exp merge with the gated residual mass (mode 0), or the gate
// mixture of the separately normalised branches (mode 1).
__global__ __launch_bounds__(kThreads) void merge_branches_kernel(const float* o_main, const float* lse_main,
                                                                  const float* o_res, const float* lse_res,
                                                                  const float* gate, float* out, int mode,
                                                                  size_t rows, int D) {
  const size_t i = blockIdx.x * (size_t)kThreads + threadIdx.x;
  if (i >= rows * D) return;
  const size_t row = i / D;
  const float g = gate[row], lm = lse_main[row], lr = lse_res[row];
  const bool has_res = lr != kNegInf;
  float v;
  if (mode == 1) {
    const float gg = has_res ? g : 0.f;
    v = (1.f - gg) * o_main[i] + gg * o_res[i];
  } else {
    const float lrg = (has_res && g > 0.f) ? lr + logf(g) : kNegInf;
    const float top = fmaxf(lm, lrg);
    const float wm = lm != kNegInf ? expf(lm - top) : 0.f;
    const float wr = lrg != kNegInf ? expf(lrg - top) : 0.f;
    const float den = wm + wr;
    v = den > 0.f ? (wm * o_main[i] + wr * o_res[i]) / den : 0.f;
  }
  out[i] = v;
}

// One block of 8 waves per (b, kv head): streams every slot of the head,
// merges the wave states in LDS, applies the gate and writes the G outputs;
// optionally appends this step's token first. Used when the (b, kv head)
// pairs alone fill the GPU, so no split-K records or second launch are needed.
// 8 waves (2 per SIMD, up to 256 registers each): every variant that needed
// more registers (a second key buffer for prefetch, or 12-16 waves) spilled
// to scratch and ran 1.5-3x slower.
constexpr int kHeadWaves = 8;
constexpr int kHeadThreads = 64 * kHeadWaves;
// Head-dependent start of the main-only blocks past the first round:
// (kStaggerMul * bh) mod kStaggerMod blocks, taken modulo their count.
constexpr int kStaggerMod = 24;
constexpr int kStaggerMul = 5;

template <typename T, int D, int GP>
__global__ __launch_bounds__(kHeadThreads) void decode_head(DecodeArgs a) {
  const int kvh = blockIdx.x, b = blockIdx.y;
  const int bh = b * a.Hkv + kvh;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hd = lane & 15, g = lane >> 4;
  T* kc = static_cast<T*>(const_cast<void*>(a.kc)) + (size_t)bh * a.C * D;
  T* vc = static_cast<T*>(const_cast<void*>(a.vc)) + (size_t)bh * a.C * D;
  const float* logc = a.logc + (size_t)bh * a.Rcap;

  // Units: the head's r + n slots (residual slots [0, r), then main slots) in
  // 64-slot blocks [64 u, 64 u + 64), each of one kind: the block holding
  // slot r, when r is not a multiple of 64, is unit u = UR - 1 for its
  // residual slots and one extra unit u = NB, dealt last, for its main slots.
  // Units go round-robin to the waves in processing order p = wave, wave + 8,
  // ..., so every wave streams about the same number of slots whatever the
  // split between the kinds, and a wave meets its residual units before its
  // main ones. The first round (p < 8) and the residual units take the
  // natural order, so a wave's first unit is slots [64 wave, 64 wave + 64)
  // (unless it is the extra unit) and its keys are requested before the
  // cache lengths are read. The main-only blocks after them start at a
  // head-dependent block and wrap around: with every head streamed from
  // slot 0 in step, some head strides put the concurrent streams of many
  // heads on the same memory channels (a 2064-slot capacity ran nearly 30%
  // slower than a 2080-slot one); staggering the heads spreads them.
  UnitRegs<T, D> ur0;
  load_unit_k<T, D>(ur0, kc, kUnit * wave, a.C - 1, hd, g, -1, nullptr);
  int r, n;
  cache_lengths(a.res_len, a.main_len, bh, a.C, a.Rcap, r, n);
  // the per-query tau of the outputs this thread finishes, requested now so
  // that the epilogue does not wait on a global load
  constexpr int kPer = (GP * D + kHeadThreads - 1) / kHeadThreads;
  float tau_q[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int h = min((tid + k * kHeadThreads) / D, a.G - 1);
    tau_q[k] = a.tau ? a.tau[(size_t)b * a.Hq + (size_t)kvh * a.G + h] : a.tau_scalar;
  }

  // fused append of this step's token as main slot r + n (Sec. 3.1): this
  // call reads it from k_new / v_new, and the wave whose unit holds it
  // stores it into the cache for later steps
  const bool app = a.k_new != nullptr && r + n < a.C;
  const int app_row = app ? r + n : -1;
  const T* kn = app ? static_cast<const T*>(a.k_new) + (size_t)bh * D : nullptr;
  const T* vn = app ? static_cast<const T*>(a.v_new) + (size_t)bh * D : nullptr;
  if (app) n += 1;

  // accumulator rows per kind, wave and query head: the residual and main
  // states side by side, so one merge pass reads both (32 KB per kind at 4
  // query heads, 128 KB at 16; one block per CU either way). A single buffer
  // reused for the main states after the residual merge cost two more
  // barriers: 24.1 -> 23.6 us per call with two buffers on the ragged GQA-7
  // batch (7 query heads per KV head).
  __shared__ float s_acc[2][kHeadWaves][GP][D];
  __shared__ float s_m[2][kHeadWaves][GP];  // per kind (0 residual, 1 main), per wave
  __shared__ float s_l[2][kHeadWaves][GP];

  Frag<T, D> q;
  if (hd < a.G) q.load(static_cast<const T*>(a.q) + ((size_t)b * a.Hq + (size_t)kvh * a.G + hd) * D, g);
  else q.zero();

  const int total = r + n;
  const int UR = (r + kUnit - 1) / kUnit, NB = (total + kUnit - 1) / kUnit;
  const bool straddle = r % kUnit != 0 && total > r;
  const int U = NB + (straddle ? 1 : 0);
  auto unit_range = [&](int u, bool& is_res, int& s0, int& end) {
    if (u < NB) {
      is_res = u < UR;
      s0 = u * kUnit;
      end = is_res ? r : total;
    } else {  // the main slots of block UR - 1
      is_res = false;
      s0 = r;
      end = min(UR * kUnit, total);
    }
  };
  WaveState<D> st;
  st.reset();
  bool in_res = true;  // wave-uniform: the residual state is not yet stored
  // one unit whose keys are already requested into ur.k
  auto run_unit = [&](int u, UnitRegs<T, D>& ur) {
    bool is_res;
    int s0, end;
    unit_range(u, is_res, s0, end);
    const int nvalid = min(kUnit, end - s0);
    if (!is_res && in_res) {
      store_wave_state<D, GP>(st, s_acc[0][wave], s_m[0][wave], s_l[0][wave], hd, g);
      st.reset();
      in_res = false;
    }
    if (is_res) load_unit_lc<T, D>(ur, logc, s0, nvalid, g);
    const bool has_app = app_row >= s0 && app_row < s0 + nvalid;
    if (has_app) {  // the new key row into the cache, from the registers that received it
#pragma unroll
      for (int t = 0; t < kTiles; ++t)
        if (s0 + 16 * t + hd == app_row) ur.k[t].store(kc + (size_t)app_row * D, g);
    }
    // the value rows are requested before the logits wait on the keys, so
    // both halves of the unit are in flight together
    load_unit_v<T, D>(ur, vc, s0, nvalid, hd, g, app_row, vn);
    float sc[kTiles][4];
    unit_logits<T, D>(ur, q, a.qk_scale, sc);
    softmax_pv<T, D>(st, ur, sc, 0, nvalid, is_res, a.beta_log2, g);
    if (has_app) {
#pragma unroll
      for (int T4 = 0; T4 < 4; ++T4)
#pragma unroll
        for (int uu = 0; uu < 4; ++uu)
          if (s0 + 16 * T4 + 4 * g + uu == app_row)
            ur.v[4 * T4 + uu].store(vc + (size_t)app_row * D + VPiece<T, D>::kElems * hd);
    }
  };
  // processing order -> unit: blocks [lo, NB) start at block lo + ro
  const int lo = max(kHeadWaves, UR);
  const int nM = NB - lo;
  const int ro = nM > 0 ? (bh * kStaggerMul) % kStaggerMod % nM : 0;
  auto unit_of = [&](int p) {
    if (p < lo || p >= NB) return p;
    const int q = p - lo + ro;
    return lo + (q < nM ? q : q - nM);
  };
  if (wave < U) {
    bool is_res;
    int s0, end;
    unit_range(unit_of(wave), is_res, s0, end);
    if (s0 != kUnit * wave) {
      load_unit_k<T, D>(ur0, kc, s0, end - 1, hd, g, app_row, kn);
    } else if (app_row >= s0 && app_row < s0 + kUnit) {
#pragma unroll
      for (int t = 0; t < kTiles; ++t)
        if (min(s0 + 16 * t + hd, a.C - 1) == app_row) ur0.k[t].load(kn, g);
    }
    run_unit(unit_of(wave), ur0);
  }
  for (int p = wave + kHeadWaves; p < U; p += kHeadWaves) {
    const int u = unit_of(p);
    bool is_res;
    int s0, end;
    unit_range(u, is_res, s0, end);
    UnitRegs<T, D> ur;
    load_unit_k<T, D>(ur, kc, s0, end - 1, hd, g, app_row, kn);
    run_unit(u, ur);
  }
  if (in_res) {
    store_wave_state<D, GP>(st, s_acc[0][wave], s_m[0][wave], s_l[0][wave], hd, g);
    st.reset();
  }
  store_wave_state<D, GP>(st, s_acc[1][wave], s_m[1][wave], s_l[1][wave], hd, g);
  __syncthreads();

  // merge the waves' states of one kind for the outputs this thread owns:
  // max, sum and accumulator of (head h, column d) over the 8 waves
  auto merge = [&](int kind, int idx, float& M, float& l, float& o) {
    const int h = idx / D, d = idx % D;
    M = s_m[kind][0][h];
#pragma unroll
    for (int w = 1; w < kHeadWaves; ++w) M = fmaxf(M, s_m[kind][w][h]);
    o = 0.f;
    l = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int w = 0; w < kHeadWaves; ++w) {
        const float f = exp2f(s_m[kind][w][h] - M);
        o = fmaf(f, s_acc[kind][w][h][d], o);
        l = fmaf(f, s_l[kind][w][h], l);
      }
    }
  };
  float mR[kPer], lR[kPer], oR[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int idx = tid + k * kHeadThreads;
    if (idx < a.G * D) merge(0, idx, mR[k], lR[k], oR[k]);
  }
  // main states, then the gate and the shared denominator
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int idx = tid + k * kHeadThreads;
    if (idx >= a.G * D) continue;
    const int h = idx / D, d = idx % D;
    float M, l, oM;
    merge(1, idx, M, l, oM);
    // p_max = 1 / l_main (the max term is exactly 1), then the gate
    const float pmax = l > 0.f ? 1.f / l : 1.f;
    const int qh = b * a.Hq + kvh * a.G + h;
    const float g = fmaxf(a.g_min, 1.f / (1.f + expf(-(tau_q[k] - pmax) * a.alpha)));
    const float lg2g = g > 0.f ? log2f(g) : kNegInf;
    const float mRg = (mR[k] == kNegInf || lg2g == kNegInf) ? kNegInf : mR[k] + lg2g;
    const float Mx = fmaxf(M, mRg);
    const float fM = M != kNegInf ? exp2f(M - Mx) : 0.f;
    const float fR = mRg != kNegInf ? exp2f(mRg - Mx) : 0.f;
    const float den = l * fM + lR[k] * fR;
    const float num = oM * fM + oR[k] * fR;
    a.out[(size_t)qh * D + d] = den > 0.f ? num / den : 0.f;
    if (d == 0) {
      if (a.dbg_lse_main) a.dbg_lse_main[qh] = l > 0.f ? (M + log2f(l)) * kLn2 : kNegInf;
      if (a.dbg_lse_res) a.dbg_lse_res[qh] = lR[k] > 0.f ? (mR[k] + log2f(lR[k])) * kLn2 : kNegInf;
      if (a.dbg_gate) a.dbg_gate[qh] = g;
    }
  }
  if (app && tid == 0) a.main_len[bh] = n;
}

// ------------------------------------------------------ ragged schedule
//
// For batches whose (b, kv head) caches differ in length, one block per head
// leaves the CUs of short heads idle while the longest heads finish. Here the
// heads' 64-slot units form one list (per head: its residual units, then its
// main units) and block i streams units [i U / NB, (i + 1) U / NB) of it, so
// every block streams about the same number of slots; NB = max(CUs,
// ceil(U / kRagUnits)) keeps a block at <= 2 units per wave. Within a block
// unit j goes to wave j % 8; a wave keeps one online-softmax state and
// parks it in LDS slot j (the wave's first unit of that (head, kind)
// segment) when its next unit belongs to another segment, so a segment's
// states are the slots of its first (up to) 8 units. A head that lies wholly
// inside a block is finished there (gate, shared denominator); the blocks
// that share a head write partial records (per kind: max, sum, accumulator)
// and decode_ragged_combine merges them after the kernel boundary. Every
// block reads every head's lengths for the plan, so main_len is advanced by
// the combine kernel, never while a block may still read it.
constexpr int kRagUnits = 16;       // units per block at most (2 per wave)
constexpr int kRagMaxHeads = 2048;  // (b, kv head) pairs the plan holds in LDS
constexpr int kRagMinBlocks = 256;  // the chip's compute units
constexpr int kRagMaxRec = 128;     // blocks one head may span (records the combine merges)

// Head of global unit u: the last h with pre[h] <= u (pre ascending).
__device__ __forceinline__ int rag_head(const int* pre, int BH, int u) {
  int lo = 0, hi = BH - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= u) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// First unit of block b of NB over U units, and the block of unit u.
__device__ __forceinline__ int rag_lo(int b, int U, int NB) { return (int)(((long long)b * U) / NB); }
__device__ __forceinline__ int rag_block(int u, int U, int NB) {
  return (int)((((long long)u + 1) * NB - 1) / U);
}

// Units of one head: residual units, then main units (with this step's token).
__device__ __forceinline__ void rag_units(const DecodeArgs& a, int bh, int& r, int& n, int& ur, int& um, bool& app) {
  cache_lengths(a.res_len, a.main_len, bh, a.C, a.Rcap, r, n);
  app = a.k_new != nullptr && r + n < a.C;
  ur = (r + kUnit - 1) / kUnit;
  um = (n + (app ? 1 : 0) + kUnit - 1) / kUnit;
}

// Shared-softmax output of query head h from the merged main (M, l, o) and
// residual (mR, lR, oR) states of one output element (base-2 maxima), with
// the gate; returns the output and, through the references, p_max's gate.
__device__ __forceinline__ float rag_output(const DecodeArgs& a, int qh, float M, float l, float oM, float mR,
                                            float lR, float oR, float& g) {
  const float pmax = l > 0.f ? 1.f / l : 1.f;
  const float tau = a.tau ? a.tau[qh] : a.tau_scalar;
  g = fmaxf(a.g_min, 1.f / (1.f + expf(-(tau - pmax) * a.alpha)));
  const float lg2g = g > 0.f ? log2f(g) : kNegInf;
  const float mRg = (mR == kNegInf || lg2g == kNegInf) ? kNegInf : mR + lg2g;
  const float Mx = fmaxf(M, mRg);
  const float fM = M != kNegInf ? exp2f(M - Mx) : 0.f;
  const float fR = mRg != kNegInf ? exp2f(mRg - Mx) : 0.f;
  const float den = l * fM + lR * fR;
  const float num = oM * fM + oR * fR;
  return den > 0.f ? num / den : 0.f;
}

template <typename T, int D, int GP>
__global__ __launch_bounds__(kHeadThreads) void decode_ragged(DecodeArgs a) {
  __shared__ int s_pre[kRagMaxHeads];  // first unit of each head
  __shared__ int s_r[kRagMaxHeads];    // residual slots
  __shared__ int s_n[kRagMaxHeads];    // main slots, bit 30: this step's token is appended
  __shared__ int s_wsum[kHeadWaves];
  __shared__ int s_tot;
  __shared__ float s_acc[kRagUnits][GP][D];  // parked wave states, slot = relative unit
  __shared__ float s_m[kRagUnits][GP];
  __shared__ float s_l[kRagUnits][GP];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hd = lane & 15, g = lane >> 4;
  const int BH = a.BH;
  constexpr int kApp = 1 << 30;

  // plan: the heads' lengths, then the exclusive prefix of their unit counts
  // (each thread a run of consecutive heads, then a block scan of the run sums)
  const int per = (BH + kHeadThreads - 1) / kHeadThreads;
  const int h0 = min(BH, tid * per), h1 = min(BH, h0 + per);
  int run = 0;
  for (int h = h0; h < h1; ++h) {
    int r, n, ur, um;
    bool app;
    rag_units(a, h, r, n, ur, um, app);
    s_r[h] = r;
    s_n[h] = n | (app ? kApp : 0);
    s_pre[h] = ur + um;
    run += ur + um;
  }
  int incl = run;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(incl, off, 64);
    if (lane >= off) incl += v;
  }
  if (lane == 63) s_wsum[wave] = incl;
  __syncthreads();
  int before = incl - run;
  for (int w = 0; w < wave; ++w) before += s_wsum[w];
  if (tid == kHeadThreads - 1) s_tot = before + run;
  for (int h = h0; h < h1; ++h) {
    const int c = s_pre[h];
    s_pre[h] = before;
    before += c;
  }
  __syncthreads();
  const int U = s_tot;
  // at least one block per CU and at most kRagUnits units per block, but no
  // fewer than rag_min_units per block, so a head spans at most kRagMaxRec
  // blocks
  const int NB = max(1, min(max(a.rag_blocks, (U + kRagUnits - 1) / kRagUnits), U / a.rag_min_units));
  const int blk = blockIdx.x;
  if (blk == 0) {  // the plan the combine kernel reads: prefix, U, NB
    for (int h = tid; h < BH; h += kHeadThreads) a.plan[h] = s_pre[h];
    if (tid == 0) { a.plan[BH] = U; a.plan[BH + 1] = NB; }
  }
  if (blk >= NB) return;  // block-uniform
  const int lo = rag_lo(blk, U, NB), hi = rag_lo(blk + 1, U, NB);
  if (lo >= hi) return;  // fewer units than blocks: this block has none

  // this wave's units lo + wave, lo + wave + 8, ...
  WaveState<D> st;
  st.reset();
  int cur_seg = -1, cur_slot = 0, cur_bh = -1;
  Frag<T, D> q;
  for (int j = wave; j < hi - lo; j += kHeadWaves) {  // wave-uniform
    const int u = lo + j;
    const int bh = rag_head(s_pre, BH, u);
    const int r = s_r[bh], nw = s_n[bh];
    const bool app = (nw & kApp) != 0;
    const int n = nw & (kApp - 1);
    const int ur = (r + kUnit - 1) / kUnit;
    const int k = u - s_pre[bh];
    const bool is_res = k < ur;
    const int seg = 2 * bh + (is_res ? 0 : 1);
    const int nn = n + (app ? 1 : 0);
    const int s0 = is_res ? k * kUnit : r + (k - ur) * kUnit;
    const int end = is_res ? r : r + nn;
    const int nvalid = min(kUnit, end - s0);
    const int app_row = app ? r + n : -1;
    const T* kc = static_cast<const T*>(a.kc) + (size_t)bh * a.C * D;
    const T* vc = static_cast<const T*>(a.vc) + (size_t)bh * a.C * D;
    const T* kn = app ? static_cast<const T*>(a.k_new) + (size_t)bh * D : nullptr;
    const T* vn = app ? static_cast<const T*>(a.v_new) + (size_t)bh * D : nullptr;
    UnitRegs<T, D> ur_;
    load_unit_k<T, D>(ur_, kc, s0, end - 1, hd, g, app_row, kn);
    if (seg != cur_seg) {
      if (cur_seg >= 0) store_wave_state<D, GP>(st, s_acc[cur_slot], s_m[cur_slot], s_l[cur_slot], hd, g);
      st.reset();
      cur_seg = seg;
      cur_slot = j;
    }
    if (bh != cur_bh) {
      const int b = bh / a.Hkv, kvh = bh - b * a.Hkv;
      if (hd < a.G) q.load(static_cast<const T*>(a.q) + ((size_t)b * a.Hq + (size_t)kvh * a.G + hd) * D, g);
      else q.zero();
      cur_bh = bh;
    }
    if (is_res) load_unit_lc<T, D>(ur_, a.logc + (size_t)bh * a.Rcap, s0, nvalid, g);
    // the value rows are requested before the logits wait on the keys
    load_unit_v<T, D>(ur_, vc, s0, nvalid, hd, g, app_row, vn);
    float sc[kTiles][4];
    unit_logits<T, D>(ur_, q, a.qk_scale, sc);
    softmax_pv<T, D>(st, ur_, sc, 0, nvalid, is_res, a.beta_log2, g);
    if (app_row >= s0 && app_row < s0 + nvalid) {  // wave-uniform: the new rows into the cache
      constexpr int kPieces = D * (int)sizeof(T) / 16;
      if (lane < 2 * kPieces) {
        const bool isv = lane >= kPieces;
        const int c = isv ? lane - kPieces : lane;
        T* dst = static_cast<T*>(const_cast<void*>(isv ? a.vc : a.kc)) + ((size_t)bh * a.C + app_row) * D;
        reinterpret_cast<uint4*>(dst)[c] = reinterpret_cast<const uint4*>(isv ? vn : kn)[c];
      }
    }
  }
  if (cur_seg >= 0) store_wave_state<D, GP>(st, s_acc[cur_slot], s_m[cur_slot], s_l[cur_slot], hd, g);
  __syncthreads();

  // merge the parked states of each (head, kind) segment of the block; a head
  // wholly inside the block is finished here, the others leave records
  constexpr int kPer = (GP * D + kHeadThreads - 1) / kHeadThreads;
  const int hlo = rag_head(s_pre, BH, lo), hhi = rag_head(s_pre, BH, hi - 1);
  for (int bh = hlo; bh <= hhi; ++bh) {  // block-uniform
    const int r = s_r[bh], nw = s_n[bh];
    const int ur = (r + kUnit - 1) / kUnit;
    const int um = ((nw & (kApp - 1)) + ((nw & kApp) ? 1 : 0) + kUnit - 1) / kUnit;
    const int P0 = s_pre[bh];
    const bool whole = P0 >= lo && P0 + ur + um <= hi;
    const int edge = bh == hlo ? 0 : 1;
    const int b = bh / a.Hkv, kvh = bh - b * a.Hkv;
    // relative unit ranges of the two kinds inside the block
    const int ra = max(P0, lo) - lo, rb = min(P0 + ur, hi) - lo;
    const int ma = max(P0 + ur, lo) - lo, mb = min(P0 + ur + um, hi) - lo;
#pragma unroll
    for (int kk = 0; kk < kPer; ++kk) {
      const int idx = tid + kk * kHeadThreads;
      if (idx >= GP * D) continue;
      const int h = idx / D, d = idx % D;
      float Mk[2], Lk[2], Ok[2];
#pragma unroll
      for (int kind = 0; kind < 2; ++kind) {
        const int sa = kind == 0 ? ra : ma, sb = kind == 0 ? rb : mb;
        const int se = min(sa + kHeadWaves, sb);
        float M = kNegInf;
        for (int sl = sa; sl < se; ++sl) M = fmaxf(M, s_m[sl][h]);
        float l = 0.f, o = 0.f;
        if (M != kNegInf)
          for (int sl = sa; sl < se; ++sl) {
            const float f = exp2f(s_m[sl][h] - M);
            o = fmaf(f, s_acc[sl][h][d], o);
            l = fmaf(f, s_l[sl][h], l);
          }
        Mk[kind] = M; Lk[kind] = l; Ok[kind] = o;
      }
      if (whole) {
        if (h < a.G) {
          const int qh = b * a.Hq + kvh * a.G + h;
          float gg;
          a.out[(size_t)qh * D + d] = rag_output(a, qh, Mk[1], Lk[1], Ok[1], Mk[0], Lk[0], Ok[0], gg);
          if (d == 0) {
            if (a.dbg_lse_main) a.dbg_lse_main[qh] = Lk[1] > 0.f ? (Mk[1] + log2f(Lk[1])) * kLn2 : kNegInf;
            if (a.dbg_lse_res) a.dbg_lse_res[qh] = Lk[0] > 0.f ? (Mk[0] + log2f(Lk[0])) * kLn2 : kNegInf;
            if (a.dbg_gate) a.dbg_gate[qh] = gg;
          }
        }
      } else {
#pragma unroll
        for (int kind = 0; kind < 2; ++kind) {
          float* rc = a.rec + (((size_t)blk * 2 + edge) * 2 + kind) * GP * (D + 2);
          rc[h * D + d] = Ok[kind];
          if (d == 0) {
            rc[GP * D + h] = Mk[kind];
            rc[GP * D + GP + h] = Lk[kind];
          }
        }
      }
    }
  }
}

// Heads shared by several blocks: merge their records (ascending block
// order), apply the gate and write the outputs; then advance every head's
// main_len by the appended token. One block per (b, kv head). The blocks
// that share a head follow from the plan's unit count and block count alone
// (block b starts at unit b U / NB), so after the lengths and the plan the
// records' (max, sum) and the first kPF records' accumulator rows are all
// requested at once.
template <int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_ragged_combine(DecodeArgs a) {
  __shared__ int s_idx[kRagMaxRec];         // record of slot i: (block, edge), -1 if the block streamed nothing
  __shared__ float s_w[kRagMaxRec][2][GP];  // record max, then its weight e^{m - M}
  __shared__ float s_lr[kRagMaxRec][2][GP]; // record sum
  __shared__ float s_lw[2][GP];             // merged sums
  __shared__ float s_mx[2][GP];             // merged maxima
  const int bh = blockIdx.x, tid = threadIdx.x;
  int r, n, ur, um;
  bool app;
  rag_units(a, bh, r, n, ur, um, app);
  const int U = a.plan[a.BH], NB = a.plan[a.BH + 1];
  const int P0 = a.plan[bh];
  const int b0 = rag_block(P0, U, NB), b1 = rag_block(P0 + ur + um - 1, U, NB);
  const bool shared = ur + um > 0 && b0 != b1;
  constexpr int kRec = GP * (D + 2);  // floats per (block, edge, kind) record
  constexpr int kOut = (GP * D + kThreads - 1) / kThreads;
  constexpr int kPF = 8;  // records whose accumulator rows are requested together
  if (shared) {
    const int nrec = min(b1 - b0 + 1, kRagMaxRec);
    // slot i = block b0 + i; the head's first block holds it as its last
    // head unless the block starts with it; a block with an empty range left
    // no record
    for (int i = tid; i < nrec; i += kThreads) {
      const int bb = b0 + i;
      const int lo = rag_lo(bb, U, NB), hi = rag_lo(bb + 1, U, NB);
      s_idx[i] = lo < hi ? bb * 2 + (lo >= P0 ? 0 : 1) : -1;
    }
    __syncthreads();
    // every record's (max, sum) per kind and query head, and the first kPF
    // records' accumulator rows of this thread's outputs, requested together
    for (int x = tid; x < nrec * 2 * GP; x += kThreads) {
      const int i = x / (2 * GP), kind = (x / GP) % 2, h = x % GP;
      float m = kNegInf, l = 0.f;
      if (s_idx[i] >= 0) {
        const float* rc = a.rec + ((size_t)s_idx[i] * 2 + kind) * kRec;
        m = rc[GP * D + h];
        l = rc[GP * D + GP + h];
      }
      s_w[i][kind][h] = m;
      s_lr[i][kind][h] = l;
    }
    // accumulator row of slot i, kind, output (h, d): slots past nrec or of
    // blocks without a record read slot 0's record (the head's first block
    // always streamed some of it) and get weight 0
    auto acc_at = [&](int i, int kind, int h, int d) {
      const int ri = i < nrec && s_idx[i] >= 0 ? s_idx[i] : s_idx[0];
      return a.rec[((size_t)ri * 2 + kind) * kRec + h * D + d];
    };
    float pv[kOut][kPF][2];
#pragma unroll
    for (int k = 0; k < kOut; ++k) {
      const int idx = min(tid + k * kThreads, a.G * D - 1), h = idx / D, d = idx % D;
#pragma unroll
      for (int i = 0; i < kPF; ++i)
#pragma unroll
        for (int kind = 0; kind < 2; ++kind) pv[k][i][kind] = acc_at(i, kind, h, d);
    }
    __syncthreads();
    if (tid < 2 * GP) {
      const int kind = tid / GP, h = tid % GP;
      float M = kNegInf;
      for (int i = 0; i < nrec; ++i) M = fmaxf(M, s_w[i][kind][h]);
      float L = 0.f;
      for (int i = 0; i < nrec; ++i) {
        const float w = M != kNegInf && s_w[i][kind][h] != kNegInf ? exp2f(s_w[i][kind][h] - M) : 0.f;
        s_w[i][kind][h] = w;
        L = fmaf(w, s_lr[i][kind][h], L);
      }
      s_mx[kind][h] = M;
      s_lw[kind][h] = L;
    }
    __syncthreads();
    const int b = bh / a.Hkv, kvh = bh - b * a.Hkv;
#pragma unroll
    for (int k = 0; k < kOut; ++k) {
      const int idx = tid + k * kThreads;
      if (idx >= a.G * D) continue;
      const int h = idx / D, d = idx % D;
      float Ok[2] = {0.f, 0.f};
#pragma unroll
      for (int i = 0; i < kPF; ++i)
#pragma unroll
        for (int kind = 0; kind < 2; ++kind)
          if (i < nrec) Ok[kind] = fmaf(s_w[i][kind][h], pv[k][i][kind], Ok[kind]);
      for (int i0 = kPF; i0 < nrec; i0 += kPF) {  // further records, kPF at a time
        float v[kPF][2];
#pragma unroll
        for (int i = 0; i < kPF; ++i)
#pragma unroll
          for (int kind = 0; kind < 2; ++kind) v[i][kind] = acc_at(i0 + i, kind, h, d);
#pragma unroll
        for (int i = 0; i < kPF; ++i)
#pragma unroll
          for (int kind = 0; kind < 2; ++kind)
            if (i0 + i < nrec) Ok[kind] = fmaf(s_w[i0 + i][kind][h], v[i][kind], Ok[kind]);
      }
      const int qh = b * a.Hq + kvh * a.G + h;
      float gg;
      const float Mm = s_mx[1][h], Lm = s_lw[1][h], Mr = s_mx[0][h], Lr = s_lw[0][h];
      a.out[(size_t)qh * D + d] = rag_output(a, qh, Mm, Lm, Ok[1], Mr, Lr, Ok[0], gg);
      if (d == 0) {
        if (a.dbg_lse_main) a.dbg_lse_main[qh] = Lm > 0.f ? (Mm + log2f(Lm)) * kLn2 : kNegInf;
        if (a.dbg_lse_res) a.dbg_lse_res[qh] = Lr > 0.f ? (Mr + log2f(Lr)) * kLn2 : kNegInf;
        if (a.dbg_gate) a.dbg_gate[qh] = gg;
      }
    }
  }
  __syncthreads();  // every thread has read the lengths
  if (app && tid == 0) a.main_len[bh] = n + 1;
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
  if constexpr (sizeof(T) == 2 || D == 64) {  // the shapes make_decode_plan sends here
    if (pl.whole_head && !da.out_res) {
      hipLaunchKernelGGL((decode_head<T, D, GP>), dim3(pl.Hkv, pl.B), dim3(kHeadThreads), 0, stream, da);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((decode_split<T, D, GP>), dim3(pl.P, pl.Hkv, pl.B), dim3(kThreads), 0, stream, da);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = (size_t)GP * pl.P * sizeof(float);
  if (da.out_res)
    hipLaunchKernelGGL((decode_branches<D, GP>), dim3(pl.Hkv, pl.B), dim3(kThreads), lds, stream, da);
  else
    hipLaunchKernelGGL((decode_combine<D, GP>), dim3(pl.Hkv, pl.B), dim3(kThreads), lds, stream, da);
  return hipGetLastError();
}

template <typename T, int D, int GP>
hipError_t launch_ragged_typed(const RaggedPlan& pl, const DecodeArgs& da, hipStream_t stream) {
  if constexpr (GP <= 8 && (sizeof(T) == 2 || D == 64)) {
    hipLaunchKernelGGL((decode_ragged<T, D, GP>), dim3(pl.blocks), dim3(kHeadThreads), 0, stream, da);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((decode_ragged_combine<D, GP>), dim3(pl.BH), dim3(kThreads), 0, stream, da);
    return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

template <typename T, int D>
hipError_t launch_ragged_gp(const RaggedPlan& pl, const DecodeArgs& da, hipStream_t stream) {
  switch (pl.GP) {
    case 1: return launch_ragged_typed<T, D, 1>(pl, da, stream);
    case 2: return launch_ragged_typed<T, D, 2>(pl, da, stream);
    case 4: return launch_ragged_typed<T, D, 4>(pl, da, stream);
    case 8: return launch_ragged_typed<T, D, 8>(pl, da, stream);
  }
  return hipErrorInvalidValue;
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
  // one block per (b, kv head) when those alone fill the chip's CUs (fp32
  // rows of 128 take the split kernels: the head kernel would spill)
  p.whole_head = (long long)p.B * p.Hkv >= kWholeHeadMin && (s.dtype == RESKV_BF16 || p.D == 64);
  const size_t recs = (size_t)p.B * p.Hkv * p.P * p.GP;
  p.acc_off = 0;
  p.ml_off = align_up(recs * p.D * sizeof(float), 256);
  p.bytes = p.ml_off + align_up(recs * 2 * sizeof(float), 256);
  return p;
}

size_t decode_max_lds_weights() { return 48 * 1024; }

bool make_ragged_plan(const reskv_shape_t& s, RaggedPlan* plan) {
  RaggedPlan& p = *plan;
  p = RaggedPlan{};
  p.BH = s.batch * s.num_kv_heads;
  const int G = s.num_q_heads / s.num_kv_heads;
  p.GP = G <= 1 ? 1 : G <= 2 ? 2 : G <= 4 ? 4 : G <= 8 ? 8 : 16;
  if (p.GP > 8 || p.BH > kRagMaxHeads) return false;
  if (!(s.dtype == RESKV_BF16 || s.head_dim == 64)) return false;
  // a head holds at most ceil(r / 64) + ceil((C - r) / 64) <= ceil(C / 64) + 1
  // units; blocks of at least min_units units keep a head within kRagMaxRec
  // blocks, and min_units <= kRagUnits / 2 keeps every block within
  // kRagUnits units when the block count is cut to U / min_units
  const int uhead = (s.slot_cap + kUnit - 1) / kUnit + 1;
  p.min_units = (uhead + kRagMaxRec - 2) / (kRagMaxRec - 1);
  if (p.min_units > kRagUnits / 2) return false;
  const long long umax = (long long)p.BH * uhead;
  const long long nb = (umax + kRagUnits - 1) / kRagUnits;
  p.blocks = (int)(nb > kRagMinBlocks ? nb : kRagMinBlocks);
  p.plan_off = 0;
  p.rec_off = align_up((size_t)(p.BH + 2) * sizeof(int32_t), 256);
  p.bytes = p.rec_off + align_up((size_t)p.blocks * 4 * p.GP * (s.head_dim + 2) * sizeof(float), 256);
  return true;
}

hipError_t launch_decode_ragged(const reskv_shape_t& s, const reskv_gate_t& g, const RaggedPlan& pl,
                                const void* q, void* kc, void* vc, const float* logc, const int32_t* res_len,
                                int32_t* main_len, const void* k_new, const void* v_new, float* out,
                                float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate, void* workspace,
                                hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  DecodeArgs da{};
  da.k_new = k_new; da.v_new = v_new;
  da.q = q; da.kc = kc; da.vc = vc; da.logc = logc;
  da.res_len = res_len; da.main_len = main_len;
  da.plan = reinterpret_cast<int32_t*>(ws + pl.plan_off);
  da.rec = reinterpret_cast<float*>(ws + pl.rec_off);
  da.tau = g.tau; da.out = out;
  da.dbg_lse_main = dbg_lse_main; da.dbg_lse_res = dbg_lse_res; da.dbg_gate = dbg_gate;
  da.Hq = s.num_q_heads; da.Hkv = s.num_kv_heads; da.G = s.num_q_heads / s.num_kv_heads;
  da.C = s.slot_cap; da.Rcap = s.res_cap; da.BH = pl.BH; da.rag_blocks = kRagMinBlocks;
  da.rag_min_units = pl.min_units;
  da.qk_scale = kLog2e / sqrtf((float)s.head_dim);
  da.beta_log2 = g.beta * kLog2e;
  da.tau_scalar = g.tau_scalar; da.alpha = g.alpha; da.g_min = g.g_min;
  const bool bf = s.dtype == RESKV_BF16;
  if (s.head_dim == 128) return bf ? launch_ragged_gp<uint16_t, 128>(pl, da, stream) : hipErrorInvalidValue;
  if (s.head_dim == 64)
    return bf ? launch_ragged_gp<uint16_t, 64>(pl, da, stream) : launch_ragged_gp<float, 64>(pl, da, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_decode(const reskv_shape_t& s, const reskv_gate_t& g, const DecodePlan& pl,
                         const void* q, void* kc, void* vc, const float* logc,
                         const int32_t* res_len, int32_t* main_len, const void* k_new, const void* v_new,
                         float* out, float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate,
                         void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  DecodeArgs da{};
  da.k_new = k_new; da.v_new = v_new;  // appended inside the decode kernels
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

namespace {
constexpr int kMaxScratchDevices = 64;
std::once_flag g_scratch_once[kMaxScratchDevices];
void* g_scratch_ptr[kMaxScratchDevices];
hipError_t g_scratch_err[kMaxScratchDevices];
}  // namespace

hipError_t static_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  // once per device, with that device current: the address of this GPU's copy
  std::call_once(g_scratch_once[dev], [dev]() {
    void* p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? p : nullptr;
  });
  if (g_scratch_err[dev] != hipSuccess) return g_scratch_err[dev];
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_decode_branches(const reskv_shape_t& s, const reskv_gate_t& g, const DecodePlan& pl,
                                  const void* q, const void* kc, const void* vc, const float* logc,
                                  const int32_t* res_len, const int32_t* main_len, float* out_main,
                                  float* lse_main, float* out_res, float* lse_res, float* gate_out,
                                  void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  DecodeArgs da{};
  da.q = q; da.kc = kc; da.vc = vc; da.logc = logc;
  da.res_len = res_len; da.main_len = const_cast<int32_t*>(main_len);  // not written without an append
  da.part_acc = reinterpret_cast<float*>(ws + pl.acc_off);
  da.part_ml = reinterpret_cast<float*>(ws + pl.ml_off);
  da.tau = g.tau; da.out = out_main; da.out_res = out_res;
  da.dbg_lse_main = lse_main; da.dbg_lse_res = lse_res; da.dbg_gate = gate_out;
  da.Hq = pl.Hq; da.Hkv = pl.Hkv; da.G = pl.G; da.C = pl.C; da.Rcap = pl.Rcap; da.PR = pl.PR; da.P = pl.P;
  da.qk_scale = kLog2e / sqrtf((float)pl.D);
  da.beta_log2 = g.beta * kLog2e;
  da.tau_scalar = g.tau_scalar; da.alpha = g.alpha; da.g_min = g.g_min;
  const bool bf = s.dtype == RESKV_BF16;
  if (pl.D == 128) return bf ? launch_gp<uint16_t, 128>(pl, da, stream) : launch_gp<float, 128>(pl, da, stream);
  if (pl.D == 64) return bf ? launch_gp<uint16_t, 64>(pl, da, stream) : launch_gp<float, 64>(pl, da, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_merge_branches(const reskv_shape_t& s, int mode, const float* out_main, const float* lse_main,
                                 const float* out_res, const float* lse_res, const float* gate, float* out,
                                 hipStream_t stream) {
  const size_t rows = (size_t)s.batch * s.num_q_heads;
  const size_t n = rows * s.head_dim;
  hipLaunchKernelGGL(merge_branches_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                     stream, out_main, lse_main, out_res, lse_res, gate, out, mode, rows, s.head_dim);
  return hipGetLastError();
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
