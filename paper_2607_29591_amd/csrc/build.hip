// Construction of the main + residual cache of one layer (App. D, Algorithm 1
// with the residual count r given per (b, kv head)).
//
// Per (b, kv head), in launch order:
//   lse_partial    MFMA logits of the G*w observation-window rows against a
//                  256-key chunk (each wave owns 64 keys and runs over all
//                  rows); per row the max and sum of exp (base 2) over the
//                  keys it can see (causal inside the window)
//   lse_final      merges the chunk partials into one log-sum-exp per row
//   score_accum    recomputes the logits; raw[p] = sum over rows of the
//                  normalised weight of key p, for the scored positions
//   pool_scores    centred zero-padded sum (5 taps by default) over the
//                  scored positions
//   [adakv_alloc]  with cross-head allocation only: moves top-k budget
//                  between the KV heads of a sequence (one ranking of all
//                  heads' scores, per-head safeguard floor and slot cap) and
//                  rewrites each head's sizes before the selection
//   select_hist x4 radix select (4 x 8-bit digits of the fp32 bit pattern) of
//   select_count   the k_top-th and (k_top + r')-th largest score over blocks
//   select_write   of 8192 scores; ties at a threshold go to the lower
//                  position. Stable compaction writes main_idx (top-k, then
//                  the protected window), the evicted list E and the Lloyd
//                  seeds, all ascending
//   gather_init    copies the main rows into slots [r, r + m), clears the
//                  residual slots, seeds the Lloyd centres with K[seed] (fp32,
//                  bf16 hi + lo and the squared norm)
//   T x { lloyd_assign   MFMA distances ||mu||^2 - 2 k.mu with mu = hi + lo,
//                        argmin with ties to the lower centre, and per-block
//                        group histograms
//         lloyd_offsets  group starts and per-block offsets (counting sort)
//         lloyd_scatter  stable placement of E by group
//         lloyd_update   fp64 sums of the members in fixed order -> new
//                        centres; in the last round also the mean values,
//                        counts and log-counts written to the cache }
// Scores follow the SnapKV rule (App. B.2.2), selection the main-selection
// equation (Sec. 5.2), the partition objective and summaries Sec. 5.3 and
// App. B.3.
#include <math.h>

#include <vector>

#include <type_traits>

#include "common.h"
#include "internal.h"

namespace reskv {

namespace {

constexpr int kThreads = 256;
constexpr int kKeyGroups = 4;     // 256-key groups per score-pass block, one after the other
constexpr int kKeyChunk = 256 * kKeyGroups;  // keys per score-pass block
// window rows staged in LDS per scoring step: 128, or 256 when there are
// more than 128 (each key group is then loaded once for all of them)
constexpr int kRowChunk = 128;
constexpr int kRowChunkWide = 256;
// s_waitcnt immediate: vector-memory count 0, export and LDS/scalar counts
// left at their maximum (no wait on them)
constexpr int kWaitVmcnt0 = 0x0F70;
constexpr int kTokBlock = 256;     // evicted tokens per counting-sort block (histograms, scatter)
constexpr int kSelThreads = 1024;
constexpr int kSelPer = 8;                          // scores per selection thread
constexpr int kSelChunk = kSelPer * kSelThreads;   // scores per selection block
constexpr int kSelHist = 4 * 2 * 256;              // selection pass histograms per head: [pass][threshold][digit]
constexpr int kAdaThreads = 1024;

struct BuildArgs {
  const void* k;
  const void* v;
  const void* q_obs;
  void* kc;
  void* vc;
  float* logc;
  int32_t* main_idx;
  int32_t* res_len;
  int32_t* main_len;
  float* dbg_scores;
  int32_t* dbg_assign;
  float* dbg_centers;  // [T][BH][Rcap][D] or NULL
  const HeadMeta* meta;
  float2* lse_part;    // [BH][NCH][R] (max, sum) in base 2, one per lse block
  float* lse2;         // [BH][R]
  float* raw;          // [BH][S]
  float* score;        // [BH][S]
  int32_t* elist;      // [BH][S]   evicted positions, ascending
  int32_t* seeds;      // [BH][Rcap]
  float* cent;         // [BH][Rcap][D]
  uint16_t* cent_hi;   // [BH][Rcap][D]
  uint16_t* cent_lo;   // [BH][Rcap][D]
  float* cnorm;        // [BH][Rcap]
  int32_t* assign;     // [BH][S]   group of evicted token i
  int32_t* hist;       // [BH][NBLK][Rcap] block histograms -> block offsets
  int32_t* cstart;     // [BH][Rcap]
  int32_t* ccount;     // [BH][Rcap]
  int32_t* order;      // [BH][S]   evicted positions grouped by centre
  int32_t* sel_hist;   // [BH][4][2][256] selection pass histograms (zeroed by pool_scores)
  int32_t* sel_cnt;    // [BH][NSEL][4] per selection block: above / equal to each threshold
  int B, Hq, Hkv, G, C, Rcap, S, w, R, LG, NCH, NBLK, NSEL, T;
  int wr;              // leading window rows per query head that score (R = G * wr)
  int pool_half;       // pooling taps on each side of a position
  int cap_slots;       // slots a head may fill at construction (C minus the decode reserve)
  float scale2;        // log2(e) / sqrt(d)
};

// (b, kv head) of a block from blockIdx.y / .z; with rev set the heads are
// walked in the opposite order, so a kernel that re-reads the keys of the
// kernel before it starts with the heads that kernel read last (still in the
// memory-side cache) instead of the ones it read first.
__device__ __forceinline__ void block_head(const BuildArgs& a, int rev, int& b, int& kvh, int& bh) {
  bh = blockIdx.z * a.Hkv + blockIdx.y;
  if (rev) bh = a.B * a.Hkv - 1 - bh;
  b = bh / a.Hkv;
  kvh = bh - b * a.Hkv;
}

__device__ __forceinline__ float to_f32(uint16_t x) { return __uint_as_float((uint32_t)x << 16); }
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ void store_elem(uint16_t* p, float x) { *p = f32_to_bf16_rne(x); }
__device__ __forceinline__ void store_elem(float* p, float x) { *p = x; }

// Scoring row t = h*wr + i of the group: query head kvh*G + h, window row i
// (position s-w+i); only the leading wr rows of each head's window score.
// Rows [r0, r0 + nrows) are copied into LDS with rows of D*sizeof(T) + 16
// bytes (the pad keeps MFMA fragment reads free of bank conflicts); rows at
// or past R are zero.
template <typename T, int D>
__device__ __forceinline__ void stage_window_rows(unsigned char* s_q, const BuildArgs& a, int b, int kvh, int r0,
                                                  int nrows) {
  constexpr int kPieces = D * (int)sizeof(T) / 16;
  constexpr int kQRowB = D * (int)sizeof(T) + 16;
  for (int x = threadIdx.x; x < nrows * kPieces; x += blockDim.x) {
    const int rr = x / kPieces, pc = x % kPieces, t = r0 + rr;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (t < a.R) {
      const int h = t / a.wr, i = t % a.wr;
      const T* q = static_cast<const T*>(a.q_obs) + (((size_t)b * a.Hq + kvh * a.G + h) * a.w + i) * D;
      v = reinterpret_cast<const uint4*>(q)[pc];
    }
    *reinterpret_cast<uint4*>(s_q + rr * kQRowB + pc * 16) = v;
  }
}

// ---------------------------------------------------------------- scoring

// Scoring blocks stream groups of 256 keys one after the other (the lse pass
// 4, 8 or 16 groups per block as the plan chooses, the score pass 4); in each
// group a wave owns 64 keys and runs over every window row. The window rows
// are staged in LDS once per block, RC at a time: every row chunk loads the
// block's keys again, so with more than 128 rows (G w = 224, 256) the wide
// chunk of 256 rows reads each key once per pass, at two blocks per CU.

// Key fragments of the 64 keys from kw (clamped to the sequence).
template <typename T, int D>
__device__ __forceinline__ void load_score_keys(Frag<T, D> (&f)[4], const T* K, int kw, int s, int col, int grp) {
#pragma unroll
  for (int t = 0; t < 4; ++t) f[t].load(K + (size_t)min(kw + 16 * t + col, s - 1) * D, grp);
}

// lse pass: the MFMA is oriented keys x rows, C[key][row]: a lane holds 16
// keys of one row, so a row's max and sum need only two cross-lane steps.
// Each wave keeps a running (max, sum) per row over its key groups. A wave
// holds one 64-key group at a time (no second key buffer): at three waves
// per SIMD (bf16) the other blocks on the CU cover its load latency.
template <typename T, int D, int RC>
__global__ __launch_bounds__(kThreads, (RC > kRowChunk ? 2 : sizeof(T) == 2 ? 3 : 2)) void lse_partial(BuildArgs a) {
  const int ch = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  const HeadMeta hm = a.meta[bh];
  const int k0 = ch * 256 * a.LG;
  if (hm.all_main || k0 >= hm.s) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  constexpr int kQRowB = D * (int)sizeof(T) + 16;
  __shared__ __align__(16) unsigned char s_q[RC * kQRowB];
  __shared__ float2 s_ml[4][RC];
  const T* K = static_cast<const T*>(a.k) + (size_t)bh * a.S * D;
  for (int r0 = 0; r0 < a.R; r0 += RC) {
    const int nrt = (min(RC, a.R - r0) + 15) / 16;
    if (r0 > 0) __syncthreads();  // the previous chunk's rows and records are consumed
    Frag<T, D> kf[4];
    load_score_keys<T, D>(kf, K, k0 + 64 * wave, hm.s, col, grp);
    stage_window_rows<T, D>(s_q, a, b, kvh, r0, 16 * nrt);
    __syncthreads();
    // running (max, sum) of row 16 rt + col over this wave's keys, kept in
    // LDS so the row-tile loop need not be unrolled; the four lane groups
    // hold the same reduced values and each lane reads back its own writes
    for (int rt = 0; rt < nrt; ++rt) s_ml[wave][16 * rt + col] = make_float2(kNegInf, 0.f);
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);  // the first group's keys have landed
#pragma unroll 1
    for (int gi = 0; gi < a.LG; ++gi) {
      const int kw = k0 + 256 * gi + 64 * wave;  // this wave's keys in group gi
      if (gi > 0) load_score_keys<T, D>(kf, K, kw, hm.s, col, grp);
      __builtin_amdgcn_sched_barrier(0);  // the group's key loads go out before its work
      // keys up to s - w are visible to every window row (and lie below s):
      // such waves skip the per-element masks
      auto rows = [&](auto full_tag) {
        constexpr bool kFull = decltype(full_tag)::value;
#pragma unroll 1
        for (int rt = 0; rt < nrt; ++rt) {
          const int t_row = r0 + 16 * rt + col;  // window row of this lane's column
          Frag<T, D> qf;
          qf.load(reinterpret_cast<const T*>(s_q + (16 * rt + col) * kQRowB), grp);
          const int pos = t_row < a.R ? hm.s - a.w + t_row % a.wr : -1;
          // raw logits; the scale is positive, so the max commutes with it
          float v[16];
          float m = kNegInf;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const f32x4_t c = mma<D>(kf[t], qf, zero4());
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int p = kw + 16 * t + 4 * grp + i;
              const float x = (kFull || (p < hm.s && p <= pos)) ? c[i] : kNegInf;
              v[4 * t + i] = x;
              m = fmaxf(m, x);
            }
          }
          m = wave_xor_max(m, 16);
          m = wave_xor_max(m, 32);
          m = m == kNegInf ? kNegInf : m * a.scale2;
          const float2 st = s_ml[wave][16 * rt + col];
          const float m_new = fmaxf(st.x, m);
          if (m_new == kNegInf) continue;
          float l = 0.f;
#pragma unroll
          for (int j = 0; j < 16; ++j) l += fast_exp2(fmaf(v[j], a.scale2, -m_new));
          l = wave_xor_add(l, 16);
          l = wave_xor_add(l, 32);
          s_ml[wave][16 * rt + col] = make_float2(m_new, fmaf(st.y, fast_exp2(st.x - m_new), l));
        }
      };
      if (kw < hm.s) {  // wave-uniform
        if (kw + 64 <= hm.s - a.w + 1) rows(std::true_type{});
        else rows(std::false_type{});
      }

    }
    __syncthreads();
    for (int t = threadIdx.x; t < min(RC, a.R - r0); t += kThreads) {
      float M = kNegInf;
#pragma unroll
      for (int w = 0; w < 4; ++w) M = fmaxf(M, s_ml[w][t].x);
      float L = 0.f;
      if (M != kNegInf) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float2 e = s_ml[w][t];
          if (e.x != kNegInf) L = fmaf(e.y, exp2f(e.x - M), L);
        }
      }
      a.lse_part[((size_t)bh * a.NCH + ch) * a.R + r0 + t] = make_float2(M, L);
    }
  }
}

__global__ __launch_bounds__(kThreads) void lse_final(BuildArgs a) {
  const int kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  const HeadMeta hm = a.meta[bh];
  const int t = blockIdx.x * kThreads + threadIdx.x;
  if (hm.all_main || t >= a.R) return;
  const int nch = (hm.s + 256 * a.LG - 1) / (256 * a.LG);
  const float2* pp = a.lse_part + (size_t)bh * a.NCH * a.R + t;
  float M = kNegInf;
  for (int c = 0; c < nch; ++c) M = fmaxf(M, pp[(size_t)c * a.R].x);
  float L = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float2 e = pp[(size_t)c * a.R];
    if (e.x != kNegInf) L = fmaf(e.y, exp2f(e.x - M), L);
  }
  a.lse2[(size_t)bh * a.R + t] = M + log2f(L);
}

// Score pass: C[row][key]: a lane holds one key of 4 rows, so the per-key
// sums stay in registers until two final cross-lane steps, and no cross-wave
// merge is needed. One key group per wave at a time and a rolled row-tile
// loop keep it at four waves per SIMD (bf16).
template <typename T, int D, int RC>
__global__ __launch_bounds__(kThreads, (RC > kRowChunk ? 2 : sizeof(T) == 2 ? 4 : 2)) void score_accum(BuildArgs a, int rev) {
  const int ch = blockIdx.x;
  int b, kvh, bh;
  block_head(a, rev, b, kvh, bh);
  const HeadMeta hm = a.meta[bh];
  const int k0 = ch * kKeyChunk;
  if (hm.all_main || k0 >= hm.n_sc) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  constexpr int kQRowB = D * (int)sizeof(T) + 16;
  constexpr int kRT = RC / 16;
  __shared__ __align__(16) unsigned char s_q[RC * kQRowB];
  __shared__ float s_lse[RC];
  const T* K = static_cast<const T*>(a.k) + (size_t)bh * a.S * D;
  for (int r0 = 0; r0 < a.R; r0 += RC) {
    const int nr = min(RC, a.R - r0), nrt = (nr + 15) / 16;
    if (r0 > 0) __syncthreads();  // the previous chunk's rows are consumed
    Frag<T, D> kf[4];
    load_score_keys<T, D>(kf, K, k0 + 64 * wave, hm.s, col, grp);
    stage_window_rows<T, D>(s_q, a, b, kvh, r0, 16 * nrt);
    for (int t = threadIdx.x; t < nr; t += kThreads) s_lse[t] = a.lse2[(size_t)bh * a.R + r0 + t];
    __syncthreads();
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);  // the first group's keys have landed
#pragma unroll 1
    for (int gi = 0; gi < kKeyGroups; ++gi) {
      const int kw = k0 + 256 * gi + 64 * wave;  // this wave's keys in group gi
      if (gi > 0) load_score_keys<T, D>(kf, K, kw, hm.s, col, grp);
      __builtin_amdgcn_sched_barrier(0);  // the group's key loads go out before its work
      float ksum[4] = {0.f, 0.f, 0.f, 0.f};
      // keys up to s - w are visible to every window row: such waves skip the
      // per-element causal test (padded rows carry lse = +inf and add 0)
      auto rows = [&](auto full_tag) {
        constexpr bool kFull = decltype(full_tag)::value;
#pragma unroll 1
        for (int rt = 0; rt < kRT; ++rt) {
          if (rt >= nrt) break;
          Frag<T, D> qf;
          qf.load(reinterpret_cast<const T*>(s_q + (16 * rt + col) * kQRowB), grp);
          float lse[4];
          int pos[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int tl = 16 * rt + 4 * grp + i, t = r0 + tl;
            lse[i] = t < a.R ? s_lse[tl] : __builtin_huge_valf();
            pos[i] = t < a.R ? hm.s - a.w + t % a.wr : -1;  // padded rows see no key
          }
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const f32x4_t c = mma<D>(qf, kf[t], zero4());
            const int p = kw + 16 * t + col;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float e = fast_exp2(fmaf(c[i], a.scale2, -lse[i]));
              ksum[t] += (kFull || p <= pos[i]) ? e : 0.f;
            }
          }
        }
      };
      if (kw < hm.n_sc) {  // wave-uniform
        if (kw + 64 <= hm.s - a.w + 1) rows(std::true_type{});
        else rows(std::false_type{});
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          float v = ksum[t];
          v = wave_xor_add(v, 16);
          v = wave_xor_add(v, 32);
          const int p = kw + 16 * t + col;
          if (grp == 0 && p < hm.n_sc) {
            float* dst = a.raw + (size_t)bh * a.S + p;
            if (r0 == 0) *dst = v;
            else *dst += v;  // later row chunks add to this lane's own sums
          }
        }
      }

    }
  }
}

// Centred (2 * pool_half + 1)-tap sum with zero padding over the scored
// positions (5 taps for the SnapKV rule, 1 for H2O and TOVA). A thread pools
// kPoolPer consecutive positions from one window of raw scores held in
// registers (zeros outside [0, n)), adding the taps in ascending position
// order as the one-position form does.
constexpr int kPoolPer = 4;
constexpr int kPoolHalfMax = 15;  // pool_half <= 15 (pool_kernel <= 31)
__global__ __launch_bounds__(kThreads) void pool_scores(BuildArgs a) {
  const int kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  const HeadMeta hm = a.meta[bh];
  if (blockIdx.x == 0)  // the selection's pass histograms start from zero
    for (int i = threadIdx.x; i < kSelHist; i += kThreads) a.sel_hist[(size_t)bh * kSelHist + i] = 0;
  const int p0 = (blockIdx.x * kThreads + threadIdx.x) * kPoolPer;
  if (p0 >= a.S) return;
  const int n = hm.all_main ? 0 : hm.n_sc;
  const int ph = a.pool_half;
  const float* raw = a.raw + (size_t)bh * a.S;
  float w[kPoolPer + 2 * kPoolHalfMax];  // raw[p0 - kPoolHalfMax + i]
#pragma unroll
  for (int i = 0; i < kPoolPer + 2 * kPoolHalfMax; ++i) {
    const int q = p0 - kPoolHalfMax + i;
    const bool tap = q >= p0 - ph && q < p0 + kPoolPer + ph;
    w[i] = tap && q >= 0 && q < n ? raw[q] : 0.f;
  }
#pragma unroll
  for (int k = 0; k < kPoolPer; ++k) {
    const int p = p0 + k;
    if (p >= a.S) break;
    float v = -1.f;
    if (p < n) {
      v = 0.f;
#pragma unroll
      for (int j = -kPoolHalfMax; j <= kPoolHalfMax; ++j)
        if (j >= -ph && j <= ph) v += w[k + kPoolHalfMax + j];
      a.score[(size_t)bh * a.S + p] = v;
    }
    if (a.dbg_scores) a.dbg_scores[(size_t)bh * a.S + p] = v;
  }
}

// -------------------------------------------------------------- selection

// Exclusive scan of one int per thread over a block of NT threads.
template <int NT>
__device__ __forceinline__ int block_excl_scan(int v, int* s_tmp, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_tmp[wave] = x;
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int w2 = 0; w2 < NT / 64; ++w2) {
    const int t = s_tmp[w2];
    if (w2 < wave) off += t;
    tot += t;
  }
  __syncthreads();
  total = tot;
  return off + x - v;
}

// Histogram increment of bin `dig` by the lanes with `act` set. Scores share
// their leading digits (sign and exponent), so the lanes of a wave often hit
// one bin: up to two leader rounds count the lanes that share the leader's
// bin with one atomic each; the remaining lanes add their own. Called by
// every lane of the wave (act false where a lane has nothing to count).
__device__ __forceinline__ void wave_hist_add(int* hist, int dig, bool act, int lane) {
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const unsigned long long m = __ballot(act);
    if (m == 0ull) return;  // wave-uniform
    const int leader = __ffsll((long long)m) - 1;
    const int d = __shfl(dig, leader, 64);
    const unsigned long long same = __ballot(act && dig == d);
    if (lane == leader) atomicAdd(&hist[d], __popcll(same));
    act = act && dig != d;
  }
  if (act) atomicAdd(&hist[dig], 1);
}

// Selection runs over blocks of kSelChunk consecutive scores per head, so a
// head's long score list is spread over many CUs: four radix passes (8-bit
// digits, most significant first) each add the block's digit histogram of
// the scores still matching a threshold's prefix into the head's pass
// histogram; every block of the next kernel replays the digit choices from
// the completed histograms. Then the blocks count the scores above and equal
// to each threshold, and finally each block places its scores: the earlier
// blocks' counts give its output offsets and the tie ranks of its equal
// scores (ties are taken lowest position first).

// Digit of one threshold in one radix pass from its 256-bin histogram h of
// the scores matching its prefix, krem = its rank among them: the digit d and
// the count of scores in higher digits. Run by a whole wave (every lane gets
// the values).
__device__ __forceinline__ void radix_digit(const int* h, int krem, int lane, int& d, int& above) {
  // each lane holds 4 bins in descending digit order; an inclusive scan over
  // lanes gives the count of scores at or above each digit
  int c[4], own = 0;
#pragma unroll
  for (int v = 0; v < 4; ++v) { c[v] = h[255 - 4 * lane - v]; own += c[v]; }
  int incl = own;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  int run = incl - own;  // scores above this lane's first digit
  int hit_d = -1, hit_acc = 0;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    if (hit_d < 0 && run + c[v] >= krem) { hit_d = 255 - 4 * lane - v; hit_acc = run; }
    run += c[v];
  }
  // the first lane (highest digits) that reaches krem owns the digit
  const unsigned long long hit = __ballot(hit_d >= 0);
  const int src = hit ? __ffsll((long long)hit) - 1 : 63;
  d = __shfl(hit_d, src, 64);
  above = __shfl(hit_acc, src, 64);
  if (!hit) { d = 0; above = __shfl(incl, 63, 64) - h[0]; }
}

// Prefixes and remaining ranks of both thresholds (k1-th and k2-th largest)
// after radix passes [0, npass), from the head's completed pass histograms
// gh; while the two share their prefix one histogram (threshold 0's) served
// both. Run by a whole wave.
__device__ __forceinline__ void radix_replay(const int* gh, int npass, int k1, int k2, int lane, uint32_t (&pref)[2],
                                             int (&krem)[2]) {
  pref[0] = pref[1] = 0u;
  krem[0] = k1;
  krem[1] = k2;
  for (int p = 0; p < npass; ++p) {
    const int shift = 24 - 8 * p;
    const bool shared = krem[0] > 0 && krem[1] > 0 && pref[0] == pref[1];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      if (krem[q] > 0) {  // wave-uniform
        int d, above;
        radix_digit(gh + (p * 2 + (shared ? 0 : q)) * 256, krem[q], lane, d, above);
        pref[q] |= (uint32_t)d << shift;
        krem[q] -= above;
      }
    }
  }
}

// Setup shared by the selection kernels: the head's scored length, the
// block's first score and the threshold state after `npass` radix passes
// (replayed by wave 0, then read by every thread; synchronises the block).
struct SelState {
  int n, i0;
  int k1, k2;
  uint32_t pref[2];
  int krem[2];
};
__device__ __forceinline__ void sel_state(const BuildArgs& a, const HeadMeta& hm, int bh, int npass, SelState& st,
                                          int* s_gh, uint32_t* s_pref, int* s_krem) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  st.n = hm.n_sc;
  st.i0 = blockIdx.x * kSelChunk;
  st.k1 = hm.k_top;
  st.k2 = hm.k_top + hm.r_eff;
  // the completed pass histograms into LDS in one round trip, then replayed
  const int* gh = a.sel_hist + (size_t)bh * kSelHist;
  for (int x = threadIdx.x; x < npass * 512; x += blockDim.x) s_gh[x] = gh[x];
  __syncthreads();
  if (wave == 0) {
    uint32_t pf[2];
    int kr[2];
    radix_replay(s_gh, npass, st.k1, st.k2, lane, pf, kr);
    if (lane == 0) {
      s_pref[0] = pf[0]; s_pref[1] = pf[1];
      s_krem[0] = kr[0]; s_krem[1] = kr[1];
    }
  }
  __syncthreads();
  st.pref[0] = s_pref[0]; st.pref[1] = s_pref[1];
  st.krem[0] = s_krem[0]; st.krem[1] = s_krem[1];
}

// Radix pass `pass` over one block's scores: digit histograms of the scores
// matching each threshold's prefix, added into the head's pass histogram
// (zeroed by pool_scores).
__global__ __launch_bounds__(kSelThreads) void select_hist(BuildArgs a, int pass) {
  const int bh = blockIdx.z * a.Hkv + blockIdx.y;
  const HeadMeta hm = a.meta[bh];
  if (hm.all_main || (int)blockIdx.x * kSelChunk >= hm.n_sc) return;  // block-uniform
  __shared__ int s_hist[2][256];
  __shared__ int s_gh[kSelHist];
  __shared__ uint32_t s_pref[2];
  __shared__ int s_krem[2];
  const int tid = threadIdx.x, lane = tid & 63;
  for (int i = tid; i < 512; i += kSelThreads) (&s_hist[0][0])[i] = 0;
  SelState st;
  sel_state(a, hm, bh, pass, st, s_gh, s_pref, s_krem);  // synchronises the block
  if (st.krem[0] <= 0 && st.krem[1] <= 0) return;  // block-uniform
  const bool shared = st.krem[0] > 0 && st.krem[1] > 0 && st.pref[0] == st.pref[1];
  const int shift = 24 - 8 * pass;
  const uint32_t mask = pass == 0 ? 0u : ~0u << (32 - 8 * pass);
  const uint32_t* key = reinterpret_cast<const uint32_t*>(a.score + (size_t)bh * a.S);
  uint32_t u[kSelPer];
#pragma unroll
  for (int v = 0; v < kSelPer; ++v) {  // coalesced, all loads in flight together
    const int i = st.i0 + v * kSelThreads + tid;
    u[v] = i < st.n ? key[i] : 0u;
  }
#pragma unroll
  for (int v = 0; v < kSelPer; ++v) {
    const bool in = st.i0 + v * kSelThreads + tid < st.n;
    const int dig = (u[v] >> shift) & 0xff;
    wave_hist_add(s_hist[0], dig, in && st.krem[0] > 0 && (u[v] & mask) == st.pref[0], lane);
    if (!shared) wave_hist_add(s_hist[1], dig, in && st.krem[1] > 0 && (u[v] & mask) == st.pref[1], lane);
  }
  __syncthreads();
  int* gh = a.sel_hist + (size_t)bh * kSelHist + pass * 512;
  for (int x = tid; x < 512; x += kSelThreads) {
    const int c = (&s_hist[0][0])[x];
    if (c) atomicAdd(&gh[x], c);
  }
}

// Thresholds T_q = the final prefixes; krem[q] = how many scores equal to
// T_q are taken (lowest positions first); a threshold with k = 0 takes none.
// Per block: scores above and equal to each threshold.
__global__ __launch_bounds__(kSelThreads) void select_count(BuildArgs a) {
  const int bh = blockIdx.z * a.Hkv + blockIdx.y;
  const HeadMeta hm = a.meta[bh];
  if (hm.all_main || (int)blockIdx.x * kSelChunk >= hm.n_sc) return;  // block-uniform
  __shared__ int s_gh[kSelHist];
  __shared__ uint32_t s_pref[2];
  __shared__ int s_krem[2];
  SelState st;
  sel_state(a, hm, bh, 4, st, s_gh, s_pref, s_krem);
  const int tid = threadIdx.x;
  const uint32_t* key = reinterpret_cast<const uint32_t*>(a.score + (size_t)bh * a.S);
  int c[4] = {0, 0, 0, 0};  // above T1, equal T1, above T2, equal T2
#pragma unroll
  for (int v = 0; v < kSelPer; ++v) {
    const int i = st.i0 + v * kSelThreads + tid;
    if (i < st.n) {
      const uint32_t u = key[i];
      c[0] += u > st.pref[0]; c[1] += u == st.pref[0];
      c[2] += u > st.pref[1]; c[3] += u == st.pref[1];
    }
  }
  // block sums: across each wave, then the waves' partials in LDS
  __shared__ int s_part[kSelThreads / 64][4];
  const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c[q] += __shfl_xor(c[q], o, 64);
  }
  if (lane == 0)
#pragma unroll
    for (int q = 0; q < 4; ++q) s_part[wave][q] = c[q];
  __syncthreads();
  if (tid < 4) {
    int t = 0;
    for (int w = 0; w < kSelThreads / 64; ++w) t += s_part[w][tid];
    a.sel_cnt[((size_t)bh * a.NSEL + blockIdx.x) * 4 + tid] = t;
  }
}

// Placement: main_idx (top-scored, ascending, then the protected recent
// window), elist (every other scored position, ascending) and seeds (ranks
// k1 .. k2 - 1, ascending). Each thread owns kSelPer consecutive positions
// of the block's chunk and ranks them; the block's three runs are gathered
// in LDS and stored with consecutive lanes on consecutive entries.
__global__ __launch_bounds__(kSelThreads) void select_write(BuildArgs a) {
  const int bh = blockIdx.z * a.Hkv + blockIdx.y;
  const HeadMeta hm = a.meta[bh];
  const int tid = threadIdx.x, blk = blockIdx.x;
  int32_t* main_idx = a.main_idx + (size_t)bh * a.C;
  if (blk == 0 && tid == 0) {
    a.res_len[bh] = hm.r;
    a.main_len[bh] = hm.main_len;
  }
  if (hm.all_main) {
    for (int i = blk * kSelChunk + tid; i < min(hm.s, (blk + 1) * kSelChunk); i += kSelThreads) main_idx[i] = i;
    return;
  }
  // the protected recent window follows the top-scored tokens
  if (blk == 0)
    for (int i = tid; i < hm.P; i += kSelThreads) main_idx[hm.k_top + i] = hm.n_sc + i;
  if (blk * kSelChunk >= hm.n_sc) return;  // block-uniform
  __shared__ int s_gh[kSelHist];
  __shared__ uint32_t s_pref[2];
  __shared__ int s_krem[2];
  __shared__ int s_tmp[kSelThreads / 64];
  SelState st;
  sel_state(a, hm, bh, 4, st, s_gh, s_pref, s_krem);
  const uint32_t T1 = st.pref[0], T2 = st.pref[1];
  const int need1 = st.krem[0], need2 = st.krem[1];
  const bool on1 = st.k1 > 0, on2 = st.k2 > 0;
  // offsets and tie ranks from the earlier blocks' counts (full chunks)
  int base_e1 = 0, base_e2 = 0, base_top = 0, base_seed = 0;
  const int32_t* cnt = a.sel_cnt + (size_t)bh * a.NSEL * 4;
  for (int pb = 0; pb < blk; ++pb) {
    const int gt1 = cnt[4 * pb], eq1 = cnt[4 * pb + 1], gt2 = cnt[4 * pb + 2], eq2 = cnt[4 * pb + 3];
    const int top = on1 ? gt1 + min(max(need1 - base_e1, 0), eq1) : 0;
    const int sel2 = on2 ? gt2 + min(max(need2 - base_e2, 0), eq2) : 0;
    base_top += top;
    base_seed += sel2 - top;  // the top scores are among the first k2
    base_e1 += eq1;
    base_e2 += eq2;
  }
  const int base_ev = blk * kSelChunk - base_top;
  const uint32_t* key = reinterpret_cast<const uint32_t*>(a.score + (size_t)bh * a.S);
  const int lo = st.i0 + tid * kSelPer;
  uint32_t seg[kSelPer];
#pragma unroll
  for (int v = 0; v < kSelPer; ++v) seg[v] = lo + v < st.n ? key[lo + v] : 0u;
  // equal-to-threshold counts per thread, scanned: the tie ranks
  int e1 = 0, e2 = 0;
#pragma unroll
  for (int v = 0; v < kSelPer; ++v)
    if (lo + v < st.n) { e1 += (seg[v] == T1); e2 += (seg[v] == T2); }
  // both counts in one scan (each block total is at most kSelChunk < 2^16)
  int tot;
  const int eb12 = block_excl_scan<kSelThreads>(e1 | (e2 << 16), s_tmp, tot);
  const int eb1 = base_e1 + (eb12 & 0xffff), eb2 = base_e2 + (eb12 >> 16);
  auto classify = [&](uint32_t u, int& r1, int& r2, bool& top, bool& sel2) {
    top = on1 && (u > T1 || (u == T1 && r1 < need1));
    sel2 = on2 && (u > T2 || (u == T2 && r2 < need2));
    r1 += (u == T1);
    r2 += (u == T2);
  };
  int c_top = 0, c_seed = 0;
  {
    int r1 = eb1, r2 = eb2;
#pragma unroll
    for (int v = 0; v < kSelPer; ++v) {
      if (lo + v < st.n) {
        bool top, sel2;
        classify(seg[v], r1, r2, top, sel2);
        c_top += top;
        c_seed += (sel2 && !top);
      }
    }
  }
  // block-local run offsets: top-scored from the front of s_run, evicted
  // after them (the two partition the chunk), seeds in their own buffer
  // (the evicted count of the threads before this one is their positions
  // minus their top-scored ones: every earlier thread holds kSelPer)
  int nts;
  const int ots = block_excl_scan<kSelThreads>(c_top | (c_seed << 16), s_tmp, nts);
  const int n_top = nts & 0xffff, n_seed = nts >> 16;
  const int n_valid = min(kSelChunk, st.n - st.i0);
  const int n_ev = n_valid - n_top;
  int ob_top = ots & 0xffff;
  int ob_seed = ots >> 16;
  int ob_ev = n_top + min(tid * kSelPer, n_valid) - ob_top;
  __shared__ int s_run[kSelChunk];
  __shared__ int s_seed[kSelChunk];
  int r1 = eb1, r2 = eb2;
#pragma unroll
  for (int v = 0; v < kSelPer; ++v) {
    if (lo + v < st.n) {
      bool top, sel2;
      classify(seg[v], r1, r2, top, sel2);
      if (top) s_run[ob_top++] = lo + v;
      else s_run[ob_ev++] = lo + v;
      if (sel2 && !top) s_seed[ob_seed++] = lo + v;
    }
  }
  __syncthreads();
  int32_t* elist = a.elist + (size_t)bh * a.S;
  int32_t* seeds = a.seeds + (size_t)bh * a.Rcap;
  for (int i = tid; i < n_top + n_ev; i += kSelThreads) {
    if (i < n_top) main_idx[base_top + i] = s_run[i];
    else elist[base_ev + i - n_top] = s_run[i];
  }
  for (int i = tid; i < n_seed; i += kSelThreads) seeds[base_seed + i] = s_seed[i];
}

// ------------------------------------- AdaKV cross-head budget allocation

// Per sequence b (one block): the KV heads that are not all-main share their
// top-k budgets (the compared method AdaKV of App. B.2.2, which allocates
// the kept budget across heads from SnapKV scores with a safeguard
// coefficient). Head h keeps floor(safeguard * k_top_h) of its own best
// tokens; the other sum(k_top) - sum(floor) slots follow one ranking of every
// head's remaining tokens (score descending, then head, then position), a
// head taking tokens only while it holds fewer than
// cap_h = min(n_sc_h, C - r_h - P_h). A head's tokens in that ranking come
// in its own (score, position) order, so its final set is its own top-k'_h:
// only the counts k'_h are found here, and the selection then takes each
// head's top k'_h exactly as for a uniform split.
//
// With N_h(x) = the head's scored tokens above x, the ranking reaches head
// h's tokens above x after taking min(room_h, max(0, N_h(x) - floor_h)) of
// them (room_h = cap_h - floor_h). A radix search over the fp32 bit pattern
// (non-negative floats order as unsigned integers) finds the score x* of the
// last slot handed out from per-head digit histograms; the tokens tied at
// x* then go to the heads in ascending order.
__global__ __launch_bounds__(kAdaThreads) void adakv_alloc(BuildArgs a, HeadMeta* meta, double safeguard) {
  const int b = blockIdx.x, H = a.Hkv, tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  __shared__ int s_hist[kAdaMaxHeads][256];  // digit counts, then suffix sums
  __shared__ int s_floor[kAdaMaxHeads], s_room[kAdaMaxHeads], s_n[kAdaMaxHeads], s_above[kAdaMaxHeads];
  __shared__ int s_extra, s_total_room, s_digit;
  if (tid < H) {
    const HeadMeta hm = meta[b * H + tid];
    const bool live = !hm.all_main;
    const int fl = live ? (int)floor(safeguard * (double)hm.k_top) : 0;
    const int cap = live ? min(hm.n_sc, a.cap_slots - hm.r - hm.P) : 0;
    s_floor[tid] = fl;
    s_room[tid] = live ? cap - fl : 0;
    s_n[tid] = live ? hm.n_sc : 0;
    s_above[tid] = 0;
  }
  __syncthreads();
  if (tid == 0) {
    int extra = 0, room = 0;
    for (int h = 0; h < H; ++h) {
      const HeadMeta hm = meta[b * H + h];
      if (!hm.all_main) extra += hm.k_top - s_floor[h];
      room += s_room[h];
    }
    s_extra = extra;
    s_total_room = room;
    s_digit = 0;
  }
  __syncthreads();
  const int extra = s_extra;
  const bool search = extra > 0 && s_total_room > extra;  // block-uniform
  uint32_t prefix = 0u, mask = 0u;
  int digit = 0;
  for (int shift = 24; search && shift >= 0; shift -= 8) {
    for (int i = tid; i < H * 256; i += kAdaThreads) (&s_hist[0][0])[i] = 0;
    __syncthreads();
    for (int h = 0; h < H; ++h) {
      const int n = s_n[h];
      const uint32_t* key = reinterpret_cast<const uint32_t*>(a.score + ((size_t)b * H + h) * a.S);
      for (int i0 = tid; i0 < n; i0 += 4 * kAdaThreads) {
        uint32_t u[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) u[v] = i0 + v * kAdaThreads < n ? key[i0 + v * kAdaThreads] : 0u;
#pragma unroll
        for (int v = 0; v < 4; ++v)
          wave_hist_add(s_hist[h], (u[v] >> shift) & 0xff, i0 + v * kAdaThreads < n && (u[v] & mask) == prefix, lane);
      }
    }
    __syncthreads();
    // per head, suffix sums over digits: S_h[d] = tokens of the current
    // prefix range whose digit is >= d (lane l holds digits 4l .. 4l+3)
    for (int h = wave; h < H; h += kAdaThreads / 64) {
      int c[4], own = 0;
#pragma unroll
      for (int v = 0; v < 4; ++v) { c[v] = s_hist[h][4 * lane + v]; own += c[v]; }
      int incl = own;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_down(incl, o, 64);
        if (lane + o < 64) incl += y;
      }
      int run = incl - own;  // digits above this lane's four
#pragma unroll
      for (int v = 3; v >= 0; --v) { run += c[v]; s_hist[h][4 * lane + v] = run; }
    }
    __syncthreads();
    // slots handed out down to digit d: non-increasing in d, so the digits
    // reaching `extra` are a prefix 0 .. d*; their count gives d*
    bool reach = false;
    if (tid < 256) {
      long long f = 0;
      for (int h = 0; h < H; ++h) {
        const int above = s_above[h] + s_hist[h][tid] - s_floor[h];
        f += min(s_room[h], max(0, above));
      }
      reach = f >= extra;
    }
    const int cnt = __syncthreads_count(reach);
    digit = cnt > 0 ? cnt - 1 : 0;
    if (tid < H) {
      const int higher = digit < 255 ? s_hist[tid][digit + 1] : 0;
      if (shift > 0) s_above[tid] += higher;
    }
    if (tid == 0) s_digit = digit;
    prefix |= (uint32_t)digit << shift;
    mask |= 0xffu << shift;
    __syncthreads();
  }
  if (tid != 0) return;
  // counts: slots above x*, then the tokens tied at x* to the heads in order
  // (s_above counts the tokens above the last digit's range, s_hist holds
  // the last digit's suffix sums)
  int rem = extra;
  int take[kAdaMaxHeads];
  const int d = s_digit;
  for (int h = 0; h < H; ++h) {
    if (!search) {
      take[h] = extra == 0 ? 0 : s_room[h];
      continue;
    }
    const int gt = s_above[h] + (d < 255 ? s_hist[h][d + 1] : 0);  // tokens > x*
    take[h] = min(s_room[h], max(0, gt - s_floor[h]));
    rem -= take[h];
  }
  for (int h = 0; search && h < H; ++h) {
    const int ge = s_above[h] + s_hist[h][d];                      // tokens >= x*
    const int gt = s_above[h] + (d < 255 ? s_hist[h][d + 1] : 0);
    const int tied = max(0, ge - s_floor[h]) - max(0, gt - s_floor[h]);
    const int t = min(min(s_room[h] - take[h], tied), rem);
    take[h] += t;
    rem -= t;
  }
  for (int h = 0; h < H; ++h) {
    HeadMeta hm = meta[b * H + h];
    if (hm.all_main) continue;
    hm.k_top = s_floor[h] + take[h];
    hm.m = hm.P + hm.k_top;
    hm.main_len = hm.m;
    hm.nE = hm.s - hm.m;
    hm.r_eff = hm.r < hm.nE ? hm.r : hm.nE;
    meta[b * H + h] = hm;
  }
}

// ------------------------------------------------ gather + centre seeding

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void gather_init(BuildArgs a) {
  const int kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  const HeadMeta hm = a.meta[bh];
  constexpr int kChunks = D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  const T* K = static_cast<const T*>(a.k) + (size_t)bh * a.S * D;
  const T* V = static_cast<const T*>(a.v) + (size_t)bh * a.S * D;
  T* kc = static_cast<T*>(a.kc) + (size_t)bh * a.C * D;
  T* vc = static_cast<T*>(a.vc) + (size_t)bh * a.C * D;
  const int32_t* main_idx = a.main_idx + (size_t)bh * a.C;
  const int rows = hm.main_len + hm.r;
  for (int x = blockIdx.x * kThreads + threadIdx.x; x < rows * kChunks; x += gridDim.x * kThreads) {
    const int row = x / kChunks, ck = x % kChunks;
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    int dst;
    if (row < hm.main_len) {
      const int src = main_idx[row];
      kv = reinterpret_cast<const uint4*>(K + (size_t)src * D)[ck];
      vv = reinterpret_cast<const uint4*>(V + (size_t)src * D)[ck];
      dst = hm.r + row;
    } else {
      dst = row - hm.main_len;  // residual slot, cleared
    }
    reinterpret_cast<uint4*>(kc + (size_t)dst * D)[ck] = kv;
    reinterpret_cast<uint4*>(vc + (size_t)dst * D)[ck] = vv;
  }
  // every log-count starts empty
  for (int j = blockIdx.x * kThreads + threadIdx.x; j < a.Rcap; j += gridDim.x * kThreads)
    a.logc[(size_t)bh * a.Rcap + j] = kNegInf;
  // seeds become the first centres, one wave per centre: the fp32 copy, the
  // bf16 hi + lo split and the squared norm, summed as the update sums it (an
  // fp64 butterfly over each 64 elements, then those partials in order)
  static_assert(D % 64 == 0, "whole waves per centre row");
  const int32_t* seeds = a.seeds + (size_t)bh * a.Rcap;
  const int lane = threadIdx.x & 63;
  const int nw = gridDim.x * (kThreads / 64);
  for (int j = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6); j < hm.r_eff; j += nw) {
    const T* kr = K + (size_t)seeds[j] * D;
    const size_t ci = (size_t)bh * a.Rcap + j;
    double t = 0.0;
#pragma unroll
    for (int e0 = 0; e0 < D; e0 += 64) {
      const float x = to_f32(kr[e0 + lane]);
      const uint16_t h = f32_to_bf16_rne(x);
      a.cent[ci * D + e0 + lane] = x;
      a.cent_hi[ci * D + e0 + lane] = h;
      a.cent_lo[ci * D + e0 + lane] = f32_to_bf16_rne(x - to_f32(h));
      double sq = (double)x * x;
#pragma unroll
      for (int msk = 1; msk < 64; msk <<= 1) sq += __shfl_xor(sq, msk, 64);
      t += sq;
    }
    if (lane == 0) a.cnorm[ci] = (float)t;
  }
}

// hi = bf16(mu), lo = bf16(mu - hi), norm = ||mu||^2 (fp64 sum in a fixed
// order: a butterfly within each wave, then the waves' partials in order)
template <int D>
__device__ void prep_center(const BuildArgs& a, size_t ci, const float* mu, double* s_red) {
  static_assert(D <= kThreads, "one element per thread");
  const int tid = threadIdx.x;
  double sq = 0.0;
  if (tid < D) {
    const float x = mu[tid];
    const uint16_t h = f32_to_bf16_rne(x);
    a.cent_hi[ci * D + tid] = h;
    a.cent_lo[ci * D + tid] = f32_to_bf16_rne(x - to_f32(h));
    sq = (double)x * x;
  }
#pragma unroll
  for (int msk = 1; msk < 64; msk <<= 1) sq += __shfl_xor(sq, msk, 64);
  if ((tid & 63) == 0) s_red[tid >> 6] = sq;
  __syncthreads();
  if (tid == 0) {
    double t = 0.0;
    for (int w = 0; w < (D + 63) / 64; ++w) t += s_red[w];
    a.cnorm[ci] = (float)t;
  }
  __syncthreads();
}


// ------------------------------------------------------------------ Lloyd

// Centre fragments for one 16-centre tile: A operand rows.
template <typename T, int D>
struct CenterTile;

template <int D>
struct CenterTile<uint16_t, D> {   // split bf16: mu ~ hi + lo
  Frag<uint16_t, D> hi, lo;
};
template <int D>
struct CenterTile<float, D> {
  Frag<float, D> f;
};

// One MFMA k-step of a centre tile against one token tile (bf16: 8 elements,
// fp32: 1 element per lane).
template <int D>
__device__ __forceinline__ f32x4_t mma_step(const Frag<uint16_t, D>& c, const Frag<uint16_t, D>& t, int k,
                                            f32x4_t acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(c.w[k]), as_bf16x8(t.w[k]), acc, 0, 0, 0);
}
template <int D>
__device__ __forceinline__ f32x4_t mma_step(const Frag<float, D>& c, const Frag<float, D>& t, int k, f32x4_t acc) {
  const float4 x = c.w[k >> 2], y = t.w[k >> 2];
  const int e = k & 3;
  return __builtin_amdgcn_mfma_f32_16x16x4f32(e == 0 ? x.x : e == 1 ? x.y : e == 2 ? x.z : x.w,
                                              e == 0 ? y.x : e == 1 ? y.y : e == 2 ? y.z : y.w, acc, 0, 0, 0);
}

// Tiling of the assignment. Each wave holds kTiles 16-token tiles of keys in
// registers and streams the centres from LDS; every centre fragment read from
// LDS feeds kTiles MFMAs per part (hi and lo for bf16), so LDS traffic per
// MFMA falls as 1 / kTiles. bf16: 4 tiles (64 tokens per wave) in blocks of 4
// waves at four waves per SIMD, so four blocks share a CU and drift out of
// step: some load keys while others run MFMAs. At d = 128 the kernel with the
// lo part stages 16 centres at a time, which keeps it within the 128
// registers of that occupancy. fp32 (twice the key registers): 2 tiles,
// 8 waves, four waves per SIMD. Histograms stay per 256-token block of the
// evicted list.
template <typename T, int D, bool kLo>
struct AssignShape {
  static constexpr bool kBf = sizeof(T) == 2;
  static constexpr int kTiles = kBf ? 4 : 2;
  static constexpr int kWaves = kBf ? 4 : 8;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kWavesPerSimd = 4;
  static constexpr int kCenters = kBf ? (kLo && D == 128 ? 16 : 32) : 64;  // centres staged in LDS per step
  static constexpr int kTokens = kWaves * 16 * kTiles;                    // evicted tokens per block
  static constexpr int kSubs = kTokens / kTokBlock;                       // histogram blocks per block
  static_assert(kTokens % kTokBlock == 0, "assignment tiling");
};

// Assignment of AssignShape::kTokens evicted tokens to the nearest centre:
// C[centre][token] = mu.k on MFMA with mu = hi + lo (bf16 pair) or fp32,
// dist = ||mu||^2 - 2 mu.k, argmin with ties to the lower centre. All token
// tiles of a wave advance through each k-step together, so the MFMA chains
// are independent. Centres past r' are staged with an infinite norm and
// never win. kLo = false drops the lo part: the first round's centres are
// bf16 key rows, so for finite keys lo is exactly zero there and the
// distances are the same bit for bit with half the MFMAs.
template <typename T, int D, bool kLo = true>
__global__ __launch_bounds__((AssignShape<T, D, kLo>::kThreads), (AssignShape<T, D, kLo>::kWavesPerSimd)) void lloyd_assign(BuildArgs a, int iter) {
  using Shape = AssignShape<T, D, kLo>;
  constexpr bool kBf = sizeof(T) == 2;
  constexpr int kTT = Shape::kTiles;
  constexpr int kSubs = Shape::kSubs;
  constexpr int kNT = Shape::kThreads;
  constexpr int kCC = Shape::kCenters;
  constexpr int kRowB = kBf ? D * 2 + 16 : D * 4 + 16;   // padded LDS row bytes
  constexpr int kSteps = kBf ? D / 32 : D / 4;           // MFMA k-steps over the lane's share of a row
  const int blk = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  const HeadMeta hm = a.meta[bh];
  const int t0 = blk * Shape::kTokens;
  if (hm.r_eff == 0 || t0 >= hm.nE) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 15, grp = lane >> 4;
  __shared__ __align__(16) unsigned char s_c[kCC * kRowB * (kBf ? 2 : 1)];
  __shared__ float s_norm[kCC];
  extern __shared__ int s_hist[];  // [r_eff]: one 256-token histogram block at a time

  const T* K = static_cast<const T*>(a.k) + (size_t)bh * a.S * D;
  const int32_t* elist = a.elist + (size_t)bh * a.S;
  const int tw = t0 + wave * 16 * kTT;  // this wave's first token
  Frag<T, D> tk[kTT];
#pragma unroll
  for (int tt = 0; tt < kTT; ++tt) {
    const int i = min(tw + 16 * tt + col, hm.nE - 1);
    tk[tt].load(K + (size_t)elist[i] * D, grp);
  }
  // per token tile: the lane's best distance and centre (over the centres of
  // its lane group, merged across the groups at the end)
  float best[kTT];
  int bidx[kTT];
#pragma unroll
  for (int tt = 0; tt < kTT; ++tt) { best[tt] = __builtin_huge_valf(); bidx[tt] = 0x7fffffff; }

  const size_t cbase = (size_t)bh * a.Rcap;
  // centre chunks are staged through one LDS buffer; the next chunk's global
  // loads are issued before this chunk's MFMAs and written after a barrier
  constexpr int kPieces = (kBf ? D * 2 : D * 4) / 16;       // 16-byte pieces per row
  constexpr int kPer = kCC * kPieces / kNT;   // pieces per thread
  static_assert(kCC * kPieces % kNT == 0, "staging split");
  uint4 ph[kPer], pl[kPer];
  float pn = 0.f;
  auto fetch = [&](int j0) {
    const int nj = min(kCC, hm.r_eff - j0);
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int x = tid + u * kNT, jj = x / kPieces, pc = x % kPieces;
      ph[u] = pl[u] = make_uint4(0, 0, 0, 0);
      if (jj < nj) {
        if (kBf) {
          ph[u] = reinterpret_cast<const uint4*>(a.cent_hi + (cbase + j0 + jj) * D)[pc];
          if (kLo) pl[u] = reinterpret_cast<const uint4*>(a.cent_lo + (cbase + j0 + jj) * D)[pc];
        } else {
          ph[u] = reinterpret_cast<const uint4*>(a.cent + (cbase + j0 + jj) * D)[pc];
        }
      }
    }
    if (tid < kCC) pn = tid < nj ? a.cnorm[cbase + j0 + tid] : __builtin_huge_valf();
  };
  auto commit = [&]() {
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int x = tid + u * kNT, jj = x / kPieces, pc = x % kPieces;
      *reinterpret_cast<uint4*>(s_c + jj * kRowB + pc * 16) = ph[u];
      if (kBf && kLo) *reinterpret_cast<uint4*>(s_c + (kCC + jj) * kRowB + pc * 16) = pl[u];
    }
    if (tid < kCC) s_norm[tid] = pn;
  };
  fetch(0);
  commit();
  for (int j0 = 0; j0 < hm.r_eff; j0 += kCC) {
    const int nj = min(kCC, hm.r_eff - j0);
    __syncthreads();  // the chunk in LDS is complete
    if (j0 + kCC < hm.r_eff) fetch(j0 + kCC);
    const int nct = (nj + 15) / 16;
    for (int ct = 0; ct < nct; ++ct) {  // block-uniform
      const int crow = 16 * ct + col;
      f32x4_t acc[kTT];
#pragma unroll
      for (int tt = 0; tt < kTT; ++tt) acc[tt] = zero4();
      if constexpr (kBf) {
        // one k-step of the hi and lo centre rows at a time: 8 elements per
        // lane, the same pieces as the token fragments (Frag layout)
        const unsigned char* rh = s_c + crow * kRowB + 16 * grp;
        const unsigned char* rl = s_c + (kCC + crow) * kRowB + 16 * grp;
#pragma unroll
        for (int k = 0; k < kSteps; ++k) {
          const uint4 ch = *reinterpret_cast<const uint4*>(rh + 64 * k);
          const uint4 cl = kLo ? *reinterpret_cast<const uint4*>(rl + 64 * k) : make_uint4(0, 0, 0, 0);
#pragma unroll
          for (int tt = 0; tt < kTT; ++tt)
            acc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ch), as_bf16x8(tk[tt].w[k]), acc[tt], 0, 0, 0);
          if constexpr (kLo) {
#pragma unroll
            for (int tt = 0; tt < kTT; ++tt)
              acc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cl), as_bf16x8(tk[tt].w[k]), acc[tt], 0, 0, 0);
          }
        }
      } else {
        Frag<T, D> ch;
        ch.load(reinterpret_cast<const T*>(s_c + crow * kRowB), grp);
#pragma unroll
        for (int k = 0; k < kSteps; ++k)
#pragma unroll
          for (int tt = 0; tt < kTT; ++tt) acc[tt] = mma_step<D>(ch, tk[tt], k, acc[tt]);
      }
      float nrm[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) nrm[i] = s_norm[16 * ct + 4 * grp + i];
      const int jb = j0 + 16 * ct + 4 * grp;
      // the lane's 4 centres in ascending order, then against earlier
      // tiles; each step runs for all token tiles before the next, so the
      // tiles' independent compare-select chains interleave
      float bv[kTT];
      int bi[kTT];
#pragma unroll
      for (int tt = 0; tt < kTT; ++tt) {
        bv[tt] = fmaf(-2.f, acc[tt][0], nrm[0]);
        bi[tt] = jb;
      }
#pragma unroll
      for (int i = 1; i < 4; ++i)
#pragma unroll
        for (int tt = 0; tt < kTT; ++tt) {
          const float dist = fmaf(-2.f, acc[tt][i], nrm[i]);
          const bool lt = dist < bv[tt];
          bi[tt] = lt ? jb + i : bi[tt];
          bv[tt] = lt ? dist : bv[tt];
        }
#pragma unroll
      for (int tt = 0; tt < kTT; ++tt) {
        const bool lt = bv[tt] < best[tt];
        bidx[tt] = lt ? bi[tt] : bidx[tt];
        best[tt] = lt ? bv[tt] : best[tt];
      }
    }
    if (j0 + kCC < hm.r_eff) {  // block-uniform
      __syncthreads();  // every wave is done with this chunk
      commit();
    }
  }
  // argmin across the 4 lane groups (centres interleave across them): ties
  // to the lower index
#pragma unroll
  for (int tt = 0; tt < kTT; ++tt) {
    float bv = best[tt];
    int bi = bidx[tt];
#pragma unroll
    for (int msk = 16; msk < 64; msk <<= 1) {
      const float ov = __shfl_xor(bv, msk, 64);
      const int oi = __shfl_xor(bi, msk, 64);
      if (ov < bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
    }
    if (bi >= hm.r_eff) bi = 0;  // only reachable with non-finite keys
    bidx[tt] = bi;
    const int i = tw + 16 * tt + col;
    if (grp == 0 && i < hm.nE) {
      a.assign[(size_t)bh * a.S + i] = bi;
      if (a.dbg_assign) a.dbg_assign[((size_t)iter * a.B * a.Hkv + bh) * a.S + elist[i]] = bi;
    }
  }
  // group histograms of the 256-token blocks of the evicted list that this
  // block covers and that hold tokens, one at a time through LDS
  for (int q = 0; q < kSubs && t0 + q * kTokBlock < hm.nE; ++q) {  // block-uniform
    for (int j = tid; j < hm.r_eff; j += kNT) s_hist[j] = 0;
    __syncthreads();
#pragma unroll
    for (int tt = 0; tt < kTT; ++tt) {
      const int i = tw + 16 * tt + col;
      if (grp == 0 && i < hm.nE && (i - t0) / kTokBlock == q) atomicAdd(&s_hist[bidx[tt]], 1);
    }
    __syncthreads();
    int32_t* hist = a.hist + ((size_t)bh * a.NBLK + blk * kSubs + q) * a.Rcap;
    for (int j = tid; j < hm.r_eff; j += kNT) hist[j] = s_hist[j];
    __syncthreads();
  }
}

// Group sizes and counting-sort offsets: hist[blk][j] becomes the first
// output position of block blk's members of group j. One 1024-thread block
// per head; the groups take `cols` threads (r' rounded up to a power of two,
// at most 1024) and the histogram rows are split among the 1024 / cols row
// groups, so a head with few groups still has every thread walking rows.
constexpr int kOffThreads = 1024;
__global__ __launch_bounds__(kOffThreads) void lloyd_offsets(BuildArgs a) {
  const int kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  const HeadMeta hm = a.meta[bh];
  if (hm.r_eff == 0) return;
  __shared__ int s_part[kOffThreads];   // per (row group, group) row sums
  __shared__ int s_start[kOffThreads];  // first output position of each group
  __shared__ int s_tmp[kOffThreads / 64];
  const int nblk = (hm.nE + kTokBlock - 1) / kTokBlock;
  int32_t* hist = a.hist + (size_t)bh * a.NBLK * a.Rcap;
  int cols = 1;
  while (cols < hm.r_eff && cols < kOffThreads) cols <<= 1;
  const int ngrp = kOffThreads / cols;
  const int c = threadIdx.x % cols, rg = threadIdx.x / cols;
  const int per = (nblk + ngrp - 1) / ngrp;
  const int q_lo = min(nblk, rg * per), q_hi = min(nblk, q_lo + per);
  // the rows of this thread's range are read in batches of kBatch independent
  // loads so the walk is not a chain of memory round trips
  constexpr int kBatch = 16;
  int carry = 0;
  for (int j0 = 0; j0 < hm.r_eff; j0 += cols) {
    const int j = j0 + c;
    const bool act = j < hm.r_eff;
    int tot = 0;
    if (act) {
      for (int q0 = q_lo; q0 < q_hi; q0 += kBatch) {
        int v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) v[u] = q0 + u < q_hi ? hist[(size_t)(q0 + u) * a.Rcap + j] : 0;
#pragma unroll
        for (int u = 0; u < kBatch; ++u) tot += v[u];
      }
    }
    s_part[threadIdx.x] = tot;
    __syncthreads();
    int before = 0, col_tot = 0;  // rows of lower row groups come first
    for (int g2 = 0; g2 < ngrp; ++g2) {
      const int v = s_part[g2 * cols + c];
      before += g2 < rg ? v : 0;
      col_tot += v;
    }
    int all;
    const int start = carry + block_excl_scan<kOffThreads>(rg == 0 && act ? col_tot : 0, s_tmp, all);
    if (rg == 0) s_start[c] = start;  // the row-group-0 threads come first in the scan
    __syncthreads();
    if (act) {
      const int first = s_start[c];
      if (rg == 0) {
        a.cstart[(size_t)bh * a.Rcap + j] = first;
        a.ccount[(size_t)bh * a.Rcap + j] = col_tot;
      }
      int run = first + before;
      for (int q0 = q_lo; q0 < q_hi; q0 += kBatch) {
        int v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) v[u] = q0 + u < q_hi ? hist[(size_t)(q0 + u) * a.Rcap + j] : 0;
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          if (q0 + u < q_hi) hist[(size_t)(q0 + u) * a.Rcap + j] = run;
          run += v[u];
        }
      }
    }
    carry += all;
    __syncthreads();  // s_part and s_start are rewritten by the next pass
  }
}

// Stable placement: members of a group keep ascending evicted order. A
// token's rank inside its 256-token block is the number of earlier tokens
// there in the same group: within a wave, the lanes sharing its group come
// from one ballot per bit of the group index; across the block's waves, from
// a per-wave count table in LDS (dynamic, kTokBlock / 64 rows of r' ints).
__global__ __launch_bounds__(kTokBlock) void lloyd_scatter(BuildArgs a) {
  const int blk = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  const HeadMeta hm = a.meta[bh];
  const int t0 = blk * kTokBlock;
  if (hm.r_eff == 0 || t0 >= hm.nE) return;
  constexpr int kNW = kTokBlock / 64;
  extern __shared__ int s_cnt[];  // [kNW][r_eff]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = t0 + tid;
  const bool live = i < hm.nE;
  const int g = live ? a.assign[(size_t)bh * a.S + i] : 0;
  const int src = live ? a.elist[(size_t)bh * a.S + i] : 0;
  for (int j = tid; j < kNW * hm.r_eff; j += kTokBlock) s_cnt[j] = 0;
  uint64_t peers = __ballot(live);
  const int nbits = hm.r_eff > 1 ? 32 - __clz(hm.r_eff - 1) : 0;
  for (int bit = 0; bit < nbits; ++bit) {
    const bool on = (g >> bit) & 1;
    const uint64_t set = __ballot(live && on);
    peers &= on ? set : ~set;
  }
  const int in_wave = __popcll(peers & ((1ull << lane) - 1));
  __syncthreads();  // the table is cleared
  if (live && in_wave == 0) s_cnt[wave * hm.r_eff + g] = __popcll(peers);
  __syncthreads();
  if (!live) return;
  int rank = in_wave;
  for (int w = 0; w < wave; ++w) rank += s_cnt[w * hm.r_eff + g];
  const int dst = a.hist[((size_t)bh * a.NBLK + blk) * a.Rcap + g] + rank;
  a.order[(size_t)bh * a.S + dst] = src;
}

// Member indices q, q + NG, q + 2NG, q + 3NG of a group's sorted list.
__device__ __forceinline__ void load_ids(int (&id)[4], const int32_t* mem, int q, int NG) {
#pragma unroll
  for (int u = 0; u < 4; ++u) id[u] = mem[q + u * NG];
}

// New centre of group j = fp64 mean of its members' keys, summed in a fixed
// order; an empty group keeps its centre. The last round also writes the
// entry: mean key and mean value in the cache dtype, and log c_j. Each
// thread keeps four member rows in flight and requests the next four
// members' indices right behind them, so a long group (the first round's
// groups, grown around single seed keys, run from a few rows to thousands)
// waits one memory round trip per step. bf16 rows stay packed until they are
// added (68 registers, seven blocks per CU).
// kKV (last round, bf16): each member's key and value rows are read in the
// same loop, twice the rows in flight of two passes one after the other.
template <typename T, int D, bool kKV = false>
__global__ __launch_bounds__(kThreads, (kKV && sizeof(T) == 2 ? 4 : sizeof(T) == 2 ? 7 : 4)) void lloyd_update(BuildArgs a, int last, int rev) {
  const int j = blockIdx.x;
  int b, kvh, bh;
  block_head(a, rev, b, kvh, bh);
  const HeadMeta hm = a.meta[bh];
  if (j >= hm.r_eff) return;
  constexpr int CPR = D / 8;            // lanes per row, 8 elements each
  constexpr int NG = kThreads / CPR;    // member groups
  __shared__ double s_sum[NG][D];
  __shared__ float s_mu[D];
  __shared__ double s_red[D];
  const int tid = threadIdx.x, c = tid % CPR, g = tid / CPR;
  const size_t ci = (size_t)bh * a.Rcap + j;
  const int cnt = a.ccount[ci];
  const int32_t* mem = a.order + (size_t)bh * a.S + a.cstart[ci];
  const T* K = static_cast<const T*>(a.k) + (size_t)bh * a.S * D;
  const T* V = static_cast<const T*>(a.v) + (size_t)bh * a.S * D;
  if constexpr (kKV && sizeof(T) == 2) {
    // last round: the key and value rows of each member are read together
    // (twice the rows in flight), each summed in member order as below
    double ak[8], av[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) ak[e] = av[e] = 0.0;
    auto add8 = [](double (&acc)[8], const uint4& w) {
      const uint32_t pw[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] += (double)bf16_lo(pw[e]);
        acc[2 * e + 1] += (double)bf16_hi(pw[e]);
      }
    };
    int q = g;
    int id[4];
    if (q + 3 * NG < cnt) load_ids(id, mem, q, NG);
    for (; q + 3 * NG < cnt; q += 4 * NG) {
      uint4 wk[4], wv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const size_t off = (size_t)id[u] * D + 8 * c;
        wk[u] = *reinterpret_cast<const uint4*>(K + off);
        wv[u] = *reinterpret_cast<const uint4*>(V + off);
      }
      if (q + 7 * NG < cnt) load_ids(id, mem, q + 4 * NG, NG);  // the next rows' indices
#pragma unroll
      for (int u = 0; u < 4; ++u) add8(ak, wk[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u) add8(av, wv[u]);
    }
    for (; q < cnt; q += NG) {
      const size_t off = (size_t)mem[q] * D + 8 * c;
      const uint4 wk = *reinterpret_cast<const uint4*>(K + off);
      const uint4 wv = *reinterpret_cast<const uint4*>(V + off);
      add8(ak, wk);
      add8(av, wv);
    }
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
      for (int e = 0; e < 8; ++e) s_sum[g][8 * c + e] = pass == 0 ? ak[e] : av[e];
      __syncthreads();
      if (tid < D) {
        double t = 0.0;
        for (int gg = 0; gg < NG; ++gg) t += s_sum[gg][tid];
        const float mean = cnt > 0 ? (float)(t / cnt) : 0.f;
        if (pass == 0) {
          const float mu = cnt > 0 ? mean : a.cent[ci * D + tid];  // empty group keeps its centre
          a.cent[ci * D + tid] = mu;
          store_elem(static_cast<T*>(a.kc) + ((size_t)bh * a.C + j) * D + tid, mu);
        } else {
          store_elem(static_cast<T*>(a.vc) + ((size_t)bh * a.C + j) * D + tid, mean);
        }
      }
      __syncthreads();
    }
    if (tid == 0) a.logc[ci] = cnt > 0 ? logf((float)cnt) : kNegInf;
    return;
  }
  for (int pass = 0; pass < (last ? 2 : 1); ++pass) {
    const T* X = pass == 0 ? K : V;
    double acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0;
    // members g, g + NG, g + 2NG, ... in order; four 16-byte row loads in
    // flight, and (wider variant) the next four members' indices requested
    // behind them; the packed variant has no registers to spare for them
    int q = g;
    int id[4];
    if (q + 3 * NG < cnt) load_ids(id, mem, q, NG);
    for (; q + 3 * NG < cnt; q += 4 * NG) {
      if constexpr (sizeof(T) == 2) {  // rows stay packed until added: 4 registers each
        uint4 w[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) w[u] = *reinterpret_cast<const uint4*>(X + (size_t)id[u] * D + 8 * c);
        if (q + 7 * NG < cnt) load_ids(id, mem, q + 4 * NG, NG);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t pw[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[2 * e] += (double)bf16_lo(pw[e]);
            acc[2 * e + 1] += (double)bf16_hi(pw[e]);
          }
        }
      } else {
        float x[4][8];
#pragma unroll
        for (int u = 0; u < 4; ++u) load8_f32(X + (size_t)id[u] * D + 8 * c, x[u]);
        if (q + 7 * NG < cnt) load_ids(id, mem, q + 4 * NG, NG);
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[e] += (double)x[u][e];
      }
    }
    for (; q < cnt; q += NG) {
      float x[8];
      load8_f32(X + (size_t)mem[q] * D + 8 * c, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += (double)x[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) s_sum[g][8 * c + e] = acc[e];
    __syncthreads();
    if (tid < D) {
      double t = 0.0;
      for (int gg = 0; gg < NG; ++gg) t += s_sum[gg][tid];
      const float mean = cnt > 0 ? (float)(t / cnt) : 0.f;
      if (pass == 0) {
        const float mu = cnt > 0 ? mean : a.cent[ci * D + tid];  // empty group keeps its centre
        s_mu[tid] = mu;
        a.cent[ci * D + tid] = mu;
        if (last) store_elem(static_cast<T*>(a.kc) + ((size_t)bh * a.C + j) * D + tid, mu);
      } else {
        store_elem(static_cast<T*>(a.vc) + ((size_t)bh * a.C + j) * D + tid, mean);
      }
    }
    __syncthreads();
  }
  if (last) {
    if (tid == 0) a.logc[ci] = cnt > 0 ? logf((float)cnt) : kNegInf;
  } else {
    prep_center<D>(a, ci, s_mu, s_red);
  }
}

__global__ void fill_i32(int32_t* p, size_t n, int32_t v) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

// Debug export of the centres round `iter` assigns against: rows j < r' of
// the fp32 centres, zero rows after them.
__global__ __launch_bounds__(kThreads) void export_centres(BuildArgs a, int iter, int D) {
  const int kvh = blockIdx.y, b = blockIdx.z;
  const int bh = b * a.Hkv + kvh;
  const int r_eff = a.meta[bh].r_eff;
  const size_t n = (size_t)a.Rcap * D;
  const float* src = a.cent + (size_t)bh * n;
  float* dst = a.dbg_centers + ((size_t)iter * a.B * a.Hkv + bh) * n;
  for (size_t i = blockIdx.x * (size_t)kThreads + threadIdx.x; i < n; i += (size_t)gridDim.x * kThreads)
    dst[i] = (int)(i / D) < r_eff ? src[i] : 0.f;
}

// Sizes of one (b, kv head) from its context length s, residual count r and
// budget b (main-selection equation, Sec. 5.2; reading R4 for |P|).
__host__ __device__ inline HeadMeta make_meta(int s, int r, int budget, int recent) {
  HeadMeta m{};
  m.s = s;
  m.r = r;
  m.m = budget - r;
  m.all_main = s <= m.m;
  m.P = m.all_main ? 0 : (recent < m.m ? recent : m.m);
  if (m.P > s) m.P = s;
  m.n_sc = m.all_main ? 0 : s - m.P;
  m.k_top = m.all_main ? 0 : m.m - m.P;
  m.nE = m.all_main ? 0 : s - m.m;
  m.r_eff = r < m.nE ? r : m.nE;
  m.main_len = m.all_main ? s : m.m;
  return m;
}

// Per-head sizes travel as kernel arguments (copied at launch), in chunks.
constexpr int kMetaChunk = 256;
struct MetaChunk {
  int first, count, recent;
  int s[kMetaChunk], r[kMetaChunk], budget[kMetaChunk];
};

__global__ void meta_kernel(HeadMeta* meta, MetaChunk c) {
  const int i = threadIdx.x;
  if (i < c.count) meta[c.first + i] = make_meta(c.s[i], c.r[i], c.budget[i], c.recent);
}

// Arguments of every construction kernel; `meta` and the outputs belong to
// the candidate being built, the scratch to the plan's workspace.
BuildArgs make_args(const BuildPlan& pl, const void* k, const void* v, const void* q_obs, const HeadMeta* meta,
                    const BuildOut& out, float* dbg_scores, int32_t* dbg_assign, float* dbg_centers,
                    void* workspace) {
  char* ws = static_cast<char*>(workspace);
  BuildArgs a{};
  a.k = k; a.v = v; a.q_obs = q_obs;
  a.kc = out.kc; a.vc = out.vc; a.logc = out.logc; a.main_idx = out.main_idx;
  a.res_len = out.res_len; a.main_len = out.main_len;
  a.dbg_scores = dbg_scores; a.dbg_assign = dbg_assign; a.dbg_centers = dbg_centers;
  a.meta = meta;
  a.lse_part = reinterpret_cast<float2*>(ws + pl.off_lsep);
  a.lse2 = reinterpret_cast<float*>(ws + pl.off_lse);
  a.raw = reinterpret_cast<float*>(ws + pl.off_raw);
  a.score = reinterpret_cast<float*>(ws + pl.off_score);
  a.elist = reinterpret_cast<int32_t*>(ws + pl.off_elist);
  a.seeds = reinterpret_cast<int32_t*>(ws + pl.off_seeds);
  a.cent = reinterpret_cast<float*>(ws + pl.off_cent);
  a.cent_hi = reinterpret_cast<uint16_t*>(ws + pl.off_chi);
  a.cent_lo = reinterpret_cast<uint16_t*>(ws + pl.off_clo);
  a.cnorm = reinterpret_cast<float*>(ws + pl.off_cnorm);
  a.assign = reinterpret_cast<int32_t*>(ws + pl.off_assign);
  a.hist = reinterpret_cast<int32_t*>(ws + pl.off_hist);
  a.cstart = reinterpret_cast<int32_t*>(ws + pl.off_cstart);
  a.ccount = reinterpret_cast<int32_t*>(ws + pl.off_ccount);
  a.order = reinterpret_cast<int32_t*>(ws + pl.off_order);
  a.sel_hist = reinterpret_cast<int32_t*>(ws + pl.off_selh);
  a.sel_cnt = reinterpret_cast<int32_t*>(ws + pl.off_selc);
  a.NSEL = pl.NSEL;
  a.B = pl.B; a.Hq = pl.Hq; a.Hkv = pl.Hkv; a.G = pl.G; a.C = pl.C; a.Rcap = pl.Rcap; a.S = pl.S; a.w = pl.w;
  a.wr = pl.wr; a.pool_half = pl.pool_half; a.R = pl.R; a.LG = pl.LG; a.NCH = pl.NCH; a.NBLK = pl.NBLK; a.T = pl.T;
  a.cap_slots = pl.C;
  a.scale2 = kLog2e / sqrtf((float)pl.D);
  return a;
}

#define RESKV_CHECK() do { e = hipGetLastError(); if (e != hipSuccess) return e; } while (0)

// The two scoring passes with RC window rows per chunk.
template <typename T, int D, int RC>
hipError_t launch_score_passes(const BuildPlan& pl, const BuildArgs& a, hipStream_t st) {
  auto grid = [&](int x) { return dim3(x < 1 ? 1 : x, pl.Hkv, pl.B); };
  hipError_t e;
  hipLaunchKernelGGL((lse_partial<T, D, RC>), grid(pl.NCH), dim3(kThreads), 0, st, a); RESKV_CHECK();
  hipLaunchKernelGGL(lse_final, grid((pl.R + kThreads - 1) / kThreads), dim3(kThreads), 0, st, a); RESKV_CHECK();
  // the second pass over the keys walks the heads in reverse (cache reuse)
  hipLaunchKernelGGL((score_accum<T, D, RC>), grid(pl.NSC), dim3(kThreads), 0, st, a, 1); RESKV_CHECK();
  return hipSuccess;
}

// Raw window scores of every scored position (lse, then weights summed).
// The wide chunk only at bf16 rows or rows of 64 (fp32 rows of 128 would
// hold one block per CU).
template <typename T, int D>
hipError_t launch_scores_typed(const BuildPlan& pl, const BuildArgs& a, hipStream_t st) {
  if constexpr (sizeof(T) == 2 || D == 64)
    if (pl.R > kRowChunk) return launch_score_passes<T, D, kRowChunkWide>(pl, a, st);
  return launch_score_passes<T, D, kRowChunk>(pl, a, st);
}

// Pooling, selection, gather and the Lloyd rounds of one candidate.
template <typename T, int D>
hipError_t launch_candidate_typed(const BuildPlan& pl, const BuildArgs& a, hipStream_t st,
                                  HeadMeta* alloc_meta = nullptr, double safeguard = 1.0) {
  const dim3 bhg(1, pl.Hkv, pl.B);
  auto grid = [&](int x) { return dim3(x < 1 ? 1 : x, pl.Hkv, pl.B); };
  hipError_t e;
  if (a.dbg_assign) {
    hipLaunchKernelGGL(fill_i32, dim3(1024), dim3(256), 0, st, a.dbg_assign,
                       (size_t)pl.T * pl.B * pl.Hkv * pl.S, -1);
    RESKV_CHECK();
  }
  hipLaunchKernelGGL(pool_scores, grid((pl.S + kThreads * kPoolPer - 1) / (kThreads * kPoolPer)), dim3(kThreads), 0,
                     st, a);
  RESKV_CHECK();
  if (alloc_meta) {
    hipLaunchKernelGGL(adakv_alloc, dim3(pl.B), dim3(kAdaThreads), 0, st, a, alloc_meta, safeguard);
    RESKV_CHECK();
  }
  for (int pass = 0; pass < 4; ++pass) {
    hipLaunchKernelGGL(select_hist, grid(pl.NSEL), dim3(kSelThreads), 0, st, a, pass);
    RESKV_CHECK();
  }
  hipLaunchKernelGGL(select_count, grid(pl.NSEL), dim3(kSelThreads), 0, st, a); RESKV_CHECK();
  hipLaunchKernelGGL(select_write, grid(pl.NSEL), dim3(kSelThreads), 0, st, a); RESKV_CHECK();
  const int rows = pl.max_main + pl.Rcap;
  const int gblocks = (rows * (D * (int)sizeof(T) / 16) + kThreads - 1) / kThreads;
  hipLaunchKernelGGL((gather_init<T, D>), grid(gblocks < 64 ? gblocks : 64), dim3(kThreads), 0, st, a);
  RESKV_CHECK();
  if (pl.max_reff > 0) {
    const size_t hist_lds = (size_t)pl.max_reff * sizeof(int);
    using S1 = AssignShape<T, D, false>;
    using S2 = AssignShape<T, D, true>;
    for (int it = 0; it < pl.T; ++it) {
      if (a.dbg_centers) {
        hipLaunchKernelGGL(export_centres, grid((pl.Rcap * D + kThreads * 8 - 1) / (kThreads * 8)), dim3(kThreads),
                           0, st, a, it, D);
        RESKV_CHECK();
      }
      if (sizeof(T) == 2 && it == 0)  // centres are the seeds' bf16 keys: lo = 0
        hipLaunchKernelGGL((lloyd_assign<T, D, false>), grid((pl.max_E + S1::kTokens - 1) / S1::kTokens),
                           dim3(S1::kThreads), hist_lds, st, a, it);
      else
        hipLaunchKernelGGL((lloyd_assign<T, D>), grid((pl.max_E + S2::kTokens - 1) / S2::kTokens), dim3(S2::kThreads),
                           hist_lds, st, a, it);
      RESKV_CHECK();
      hipLaunchKernelGGL(lloyd_offsets, bhg, dim3(kOffThreads), 0, st, a); RESKV_CHECK();
      hipLaunchKernelGGL(lloyd_scatter, grid(pl.NBLK), dim3(kTokBlock), (kTokBlock / 64) * hist_lds, st, a);
      RESKV_CHECK();
      // the update walks the heads in reverse of the assignment before and
      // after it, so each starts on the keys the other read last
      const int last = it == pl.T - 1 ? 1 : 0;
      if (last)
        hipLaunchKernelGGL((lloyd_update<T, D, true>), grid(pl.max_reff), dim3(kThreads), 0, st, a, last, 1);
      else
        hipLaunchKernelGGL((lloyd_update<T, D>), grid(pl.max_reff), dim3(kThreads), 0, st, a, last, 1);
      RESKV_CHECK();
    }
  }
  return hipSuccess;
}

#undef RESKV_CHECK

}  // namespace

void head_meta(const BuildPlan& pl, const int32_t* seq_len, const int32_t* budget, const int32_t* res_count,
               int recent, std::vector<HeadMeta>& out) {
  out.resize((size_t)pl.B * pl.Hkv);
  for (int b = 0; b < pl.B; ++b)
    for (int h = 0; h < pl.Hkv; ++h)
      out[(size_t)b * pl.Hkv + h] = make_meta(seq_len[b], res_count[b * pl.Hkv + h], budget[b], recent);
}

void init_build_plan(const reskv_shape_t& s, const reskv_build_params_t& p, BuildPlan* plan) {
  BuildPlan& pl = *plan;
  pl = BuildPlan{};
  pl.B = s.batch; pl.Hq = s.num_q_heads; pl.Hkv = s.num_kv_heads; pl.G = s.num_q_heads / s.num_kv_heads;
  pl.D = s.head_dim; pl.C = s.slot_cap; pl.Rcap = s.res_cap; pl.S = p.max_seq_len; pl.w = p.obs_window;
  pl.wr = p.fit_rows > 0 ? p.fit_rows : p.obs_window;
  pl.pool_half = (p.pool_kernel > 0 ? p.pool_kernel : 5) / 2;
  pl.R = pl.G * pl.wr; pl.T = p.lloyd_iters; pl.dtype = s.dtype;
}

bool fold_build_plan(const std::vector<HeadMeta>& hm, BuildPlan* plan) {
  BuildPlan& pl = *plan;
  for (const HeadMeta& m : hm) {
    if (m.s > pl.max_s) pl.max_s = m.s;
    if (m.main_len > pl.max_main) pl.max_main = m.main_len;
    if (m.r_eff > pl.max_reff) pl.max_reff = m.r_eff;
    if (m.nE > pl.max_E) pl.max_E = m.nE;
    if (m.main_len + m.r > pl.C) return false;
  }
  return true;
}

bool layout_build_plan(BuildPlan* plan) {
  BuildPlan& pl = *plan;
  if (pl.R > 1024 || pl.Rcap > 4096) return false;
  const size_t BH = (size_t)pl.B * pl.Hkv;
  // the lse pass takes 16, 8 or 4 key groups per block: the longest chunks
  // that still give at least 1024 blocks (fewer blocks write fewer partial
  // records and stage the window rows fewer times)
  pl.LG = kKeyGroups;
  for (int lg = 16; lg > kKeyGroups; lg /= 2)
    if (BH * (size_t)((pl.max_s + 256 * lg - 1) / (256 * lg)) >= 1024) {
      pl.LG = lg;
      break;
    }
  pl.NCH = (pl.max_s + 256 * pl.LG - 1) / (256 * pl.LG);
  pl.NSC = (pl.max_s + kKeyChunk - 1) / kKeyChunk;
  pl.NBLK = (pl.max_E + kTokBlock - 1) / kTokBlock;
  if (pl.NBLK < 1) pl.NBLK = 1;
  pl.NSEL = (pl.max_s + kSelChunk - 1) / kSelChunk;
  if (pl.NSEL < 1) pl.NSEL = 1;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off = align_up(off + bytes, 256); return o; };
  pl.off_meta = take(BH * sizeof(HeadMeta));
  pl.off_lsep = take(BH * pl.NCH * pl.R * sizeof(float2));
  pl.off_lse = take(BH * pl.R * sizeof(float));
  pl.off_raw = take(BH * pl.S * sizeof(float));
  pl.off_score = take(BH * pl.S * sizeof(float));
  pl.off_elist = take(BH * pl.S * sizeof(int32_t));
  pl.off_seeds = take(BH * pl.Rcap * sizeof(int32_t));
  pl.off_cent = take(BH * pl.Rcap * pl.D * sizeof(float));
  pl.off_chi = take(BH * pl.Rcap * pl.D * sizeof(uint16_t));
  pl.off_clo = take(BH * pl.Rcap * pl.D * sizeof(uint16_t));
  pl.off_cnorm = take(BH * pl.Rcap * sizeof(float));
  pl.off_assign = take(BH * pl.S * sizeof(int32_t));
  pl.off_hist = take(BH * pl.NBLK * pl.Rcap * sizeof(int32_t));
  pl.off_cstart = take(BH * pl.Rcap * sizeof(int32_t));
  pl.off_ccount = take(BH * pl.Rcap * sizeof(int32_t));
  pl.off_order = take(BH * pl.S * sizeof(int32_t));
  pl.off_selh = take(BH * kSelHist * sizeof(int32_t));
  pl.off_selc = take(BH * pl.NSEL * 4 * sizeof(int32_t));
  pl.bytes = off;
  return true;
}

bool make_build_plan_adakv(const reskv_shape_t& s, const reskv_build_params_t& p, double safeguard,
                           int decode_reserve, const int32_t* seq_len, const int32_t* budget,
                           const int32_t* res_count, BuildPlan* plan) {
  init_build_plan(s, p, plan);
  std::vector<HeadMeta> hm;
  head_meta(*plan, seq_len, budget, res_count, p.recent_window, hm);
  const int cslots = s.slot_cap - decode_reserve;
  for (HeadMeta& m : hm) {  // widest sizes the allocation can give each head
    if (m.all_main) continue;
    const int fl = (int)floor(safeguard * (double)m.k_top);
    const int cap = m.n_sc < cslots - m.r - m.P ? m.n_sc : cslots - m.r - m.P;
    m.main_len = m.P + cap;
    m.nE = m.s - m.P - fl;
    m.r_eff = m.r < m.nE ? m.r : m.nE;
  }
  return fold_build_plan(hm, plan) && layout_build_plan(plan);
}

bool make_build_plan(const reskv_shape_t& s, const reskv_build_params_t& p, const int32_t* seq_len,
                     const int32_t* budget, const int32_t* res_count, BuildPlan* plan) {
  init_build_plan(s, p, plan);
  std::vector<HeadMeta> hm;
  head_meta(*plan, seq_len, budget, res_count, p.recent_window, hm);
  return fold_build_plan(hm, plan) && layout_build_plan(plan);
}

hipError_t upload_meta(const BuildPlan& pl, const int32_t* seq_len, const int32_t* budget,
                       const int32_t* res_count, int recent, HeadMeta* meta, hipStream_t stream) {
  const int BH = pl.B * pl.Hkv;
  for (int first = 0; first < BH; first += kMetaChunk) {
    MetaChunk c;
    c.first = first;
    c.count = BH - first < kMetaChunk ? BH - first : kMetaChunk;
    c.recent = recent;
    for (int i = 0; i < c.count; ++i) {
      const int bh = first + i, b = bh / pl.Hkv;
      c.s[i] = seq_len[b];
      c.r[i] = res_count[bh];
      c.budget[i] = budget[b];
    }
    hipLaunchKernelGGL(meta_kernel, dim3(1), dim3(kMetaChunk), 0, stream, meta, c);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_build_scores(const BuildPlan& pl, const void* k, const void* q_obs, const HeadMeta* meta,
                               void* workspace, hipStream_t stream) {
  const BuildArgs a = make_args(pl, k, nullptr, q_obs, meta, BuildOut{}, nullptr, nullptr, nullptr, workspace);
  const bool bf = pl.dtype == RESKV_BF16;
  if (pl.D == 128) return bf ? launch_scores_typed<uint16_t, 128>(pl, a, stream) : launch_scores_typed<float, 128>(pl, a, stream);
  if (pl.D == 64) return bf ? launch_scores_typed<uint16_t, 64>(pl, a, stream) : launch_scores_typed<float, 64>(pl, a, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_build_adakv(const reskv_shape_t& s, const reskv_build_params_t& p, double safeguard,
                              int decode_reserve, const BuildPlan& pl, const void* k, const void* v,
                              const int32_t* seq_len, const void* q_obs, const int32_t* budget,
                              const int32_t* res_count, void* kc, void* vc, float* logc, int32_t* main_idx,
                              int32_t* res_len, int32_t* main_len, float* dbg_scores, int32_t* dbg_assign,
                              float* dbg_centers, void* workspace, hipStream_t stream) {
  (void)s;
  HeadMeta* meta = reinterpret_cast<HeadMeta*>(static_cast<char*>(workspace) + pl.off_meta);
  hipError_t e = upload_meta(pl, seq_len, budget, res_count, p.recent_window, meta, stream);
  if (e != hipSuccess) return e;
  e = launch_build_scores(pl, k, q_obs, meta, workspace, stream);
  if (e != hipSuccess) return e;
  const BuildOut out{kc, vc, logc, main_idx, res_len, main_len};
  BuildArgs a = make_args(pl, k, v, nullptr, meta, out, dbg_scores, dbg_assign, dbg_centers, workspace);
  a.cap_slots = pl.C - decode_reserve;
  const bool bf = pl.dtype == RESKV_BF16;
  if (pl.D == 128)
    return bf ? launch_candidate_typed<uint16_t, 128>(pl, a, stream, meta, safeguard)
              : launch_candidate_typed<float, 128>(pl, a, stream, meta, safeguard);
  if (pl.D == 64)
    return bf ? launch_candidate_typed<uint16_t, 64>(pl, a, stream, meta, safeguard)
              : launch_candidate_typed<float, 64>(pl, a, stream, meta, safeguard);
  return hipErrorInvalidValue;
}

hipError_t launch_build_candidate(const BuildPlan& pl, const void* k, const void* v, const HeadMeta* meta,
                                  const BuildOut& out, float* dbg_scores, int32_t* dbg_assign, float* dbg_centers,
                                  void* workspace, hipStream_t stream) {
  const BuildArgs a = make_args(pl, k, v, nullptr, meta, out, dbg_scores, dbg_assign, dbg_centers, workspace);
  const bool bf = pl.dtype == RESKV_BF16;
  if (pl.D == 128) return bf ? launch_candidate_typed<uint16_t, 128>(pl, a, stream) : launch_candidate_typed<float, 128>(pl, a, stream);
  if (pl.D == 64) return bf ? launch_candidate_typed<uint16_t, 64>(pl, a, stream) : launch_candidate_typed<float, 64>(pl, a, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_build(const reskv_shape_t& s, const reskv_build_params_t& p, const BuildPlan& pl,
                        const void* k, const void* v, const int32_t* seq_len, const void* q_obs,
                        const int32_t* budget, const int32_t* res_count, void* kc, void* vc,
                        float* logc, int32_t* main_idx, int32_t* res_len, int32_t* main_len,
                        float* dbg_scores, int32_t* dbg_assign, float* dbg_centers, void* workspace,
                        hipStream_t stream) {
  (void)s;
  HeadMeta* meta = reinterpret_cast<HeadMeta*>(static_cast<char*>(workspace) + pl.off_meta);
  hipError_t e = upload_meta(pl, seq_len, budget, res_count, p.recent_window, meta, stream);
  if (e != hipSuccess) return e;
  e = launch_build_scores(pl, k, q_obs, meta, workspace, stream);
  if (e != hipSuccess) return e;
  const BuildOut out{kc, vc, logc, main_idx, res_len, main_len};
  return launch_build_candidate(pl, k, v, meta, out, dbg_scores, dbg_assign, dbg_centers, workspace, stream);
}

}  // namespace reskv
