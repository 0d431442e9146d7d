// One-shot prefill compression with moment-informed selection (Sec. 5.1 prefill
// protocol; Sec. 4.2 Eq. residual; App. A.1 Eqs. app_sufficient, app_S_tilde).
//
// Stages, all on the caller's stream (H = B*Hkv heads, C = [n_s, N-w) candidates):
//   1 k_rows_cov      per (slice of 64-token tiles, head): window logits Q.K^T on MFMA,
//                     per-row online (max, sum) over the visible keys; for candidate
//                     tokens also the covariance V^T K on MFMA (tiles transposed through
//                     LDS), the sums s_k, s_v and ||v_j||.                 [reads K, V]
//   2 k_row_combine   per head: merge the row partials in slice order -> (max, 1/Z).
//   3 k_mass          per (slice, head): logits again, softmax mass summed over the
//                     window rows -> a_j, aligned chunk pooling -> abar_j,
//                     provisional score abar_j ||v_j||.                    [reads K]
//   4 k_topk          per head: radix select of the k_keep best scores, lower position
//                     first on ties; writes the kept positions in ascending order.
//   5 k_gather_rows   rows of the provisional kept set into a compact buffer.
//   6 k_cov_rows      their covariance and sums, stored negated as extra partial slots.
//   7 k_reduce        fixed-order sum of all slots = moments of the provisional evicted
//                     set; centring, clamp at tau -> S_tilde (fp32 + bf16 hi/lo), v_bar.
//   8 k_residual      per (slice, head): S_tilde k_j on MFMA, ||v_j - v_bar - c S_tilde k_j||,
//                     score_j = abar_j * that norm.                        [reads K, V]
//   9 k_topk          final kept set.
//  10 k_gather_out    retained rows (sinks, kept, window) -> k_out/v_out, idx, lens.
//  11 k_cov_rows      covariance of the final kept rows (from k_out), negated.
//  12 k_reduce        final raw moments S, s_k, s_v, n_e.
// Every reduction has a fixed order, so results are bit-reproducible.
#include "mkv_device.h"
#include "mkv_launch.h"

namespace mkv {

constexpr int TILE = 64;  // tokens per tile

__device__ __forceinline__ void store_frag(bf16_t* p, const bf16x8& f) {
  *reinterpret_cast<uint4*>(p) = __builtin_bit_cast(uint4, f);
}
__device__ __forceinline__ void store_frag(float* p, const f32x8& f) {
  reinterpret_cast<float4*>(p)[0] = make_float4(f[0], f[1], f[2], f[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(f[4], f[5], f[6], f[7]);
}

__device__ __forceinline__ void load4(const bf16_t* p, float (&o)[4]) {
  uint2 u = *reinterpret_cast<const uint2*>(p);
  o[0] = bf2f((bf16_t)(u.x & 0xffffu));
  o[1] = bf2f((bf16_t)(u.x >> 16));
  o[2] = bf2f((bf16_t)(u.y & 0xffffu));
  o[3] = bf2f((bf16_t)(u.y >> 16));
}
__device__ __forceinline__ void load4(const float* p, float (&o)[4]) {
  float4 f = *reinterpret_cast<const float4*>(p);
  o[0] = f.x; o[1] = f.y; o[2] = f.z; o[3] = f.w;
}

// Sum over the DG lanes that hold one row in the coalesced tile layout (DG = D/8).
template <int DG> __device__ __forceinline__ float row_group_sum(float x);
template <> __device__ __forceinline__ float row_group_sum<16>(float x) { return row16_sum(x); }
template <> __device__ __forceinline__ float row_group_sum<8>(float x) {
  x += __shfl_xor(x, 4);
  return quad_sum(x);
}
// Sum over the lanes of a wave that share one 8-column group (lane % DG).
template <int DG> __device__ __forceinline__ float same_group_sum(float x);
template <> __device__ __forceinline__ float same_group_sum<16>(float x) { return cross_row_sum(x); }
template <> __device__ __forceinline__ float same_group_sum<8>(float x) {
  x += __shfl_xor(x, 8);
  return cross_row_sum(x);
}

template <class T>
__device__ __forceinline__ const T* window_row(const CompressArgs& a, int head, int r) {
  const int b = head / a.Hkv, h = head % a.Hkv;
  return reinterpret_cast<const T*>(a.q_win) +
         (((size_t)b * a.Hq + (size_t)h * a.G) * a.w + r) * a.D;
}

// Covariance tile work split: D=128 -> each wave a 64x64 quadrant (4x4 MFMA tiles);
// D=64 -> each wave 16 rows x 64 columns (1x4 tiles).
template <int D> struct CovSplit {
  static constexpr int QM = D == 128 ? 4 : 1;
  static constexpr int QN = 4;
  static __device__ __forceinline__ int a0(int wave) { return D == 128 ? 64 * (wave >> 1) : 16 * wave; }
  static __device__ __forceinline__ int b0(int wave) { return D == 128 ? 64 * (wave & 1) : 0; }
};

// cacc += V_tile^T K_tile over the TILE tokens held transposed in LDS.
template <class T, int D, int LD>
__device__ __forceinline__ void cov_tile(const T (*sVT)[LD], const T (*sKT)[LD],
                                         f32x4 (&cacc)[CovSplit<D>::QM][CovSplit<D>::QN],
                                         int wave, int lane) {
  constexpr int QM = CovSplit<D>::QM, QN = CovSplit<D>::QN;
  const int a0 = CovSplit<D>::a0(wave), b0 = CovSplit<D>::b0(wave);
#pragma unroll
  for (int kk = 0; kk < TILE / 32; ++kk) {
    typename Frag<T>::type af[QM];
#pragma unroll
    for (int mi = 0; mi < QM; ++mi)
      af[mi] = load_frag(&sVT[a0 + 16 * mi + (lane & 15)][32 * kk + 8 * (lane >> 4)]);
#pragma unroll
    for (int ni = 0; ni < QN; ++ni) {
      typename Frag<T>::type bf = load_frag(&sKT[b0 + 16 * ni + (lane & 15)][32 * kk + 8 * (lane >> 4)]);
#pragma unroll
      for (int mi = 0; mi < QM; ++mi) mma(cacc[mi][ni], af[mi], bf);
    }
  }
}

// Write one slot of covariance and (s_v, s_k) partials; `sign` = -1 for downdates.
template <class T, int D>
__device__ __forceinline__ void write_cov_partials(const CompressArgs& a, int head, int slot,
                                                   f32x4 (&cacc)[CovSplit<D>::QM][CovSplit<D>::QN],
                                                   float (&sv)[8], float (&sk)[8], float sign,
                                                   float (*sRed)[2][D], int tid) {
  constexpr int QM = CovSplit<D>::QM, QN = CovSplit<D>::QN, DG = D / 8;
  const int lane = tid & 63, wave = tid >> 6;
  const int a0 = CovSplit<D>::a0(wave), b0 = CovSplit<D>::b0(wave);
  float* sp = a.spart + ((size_t)head * a.nslot + slot) * D * D;
#pragma unroll
  for (int mi = 0; mi < QM; ++mi)
#pragma unroll
    for (int ni = 0; ni < QN; ++ni)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        sp[(size_t)(a0 + 16 * mi + 4 * (lane >> 4) + i) * D + b0 + 16 * ni + (lane & 15)] =
            sign * cacc[mi][ni][i];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    sv[e] = same_group_sum<DG>(sv[e]);
    sk[e] = same_group_sum<DG>(sk[e]);
  }
  if (lane < DG) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sRed[wave][0][8 * lane + e] = sv[e];
      sRed[wave][1][8 * lane + e] = sk[e];
    }
  }
  __syncthreads();
  float* svk = a.svkpart + ((size_t)head * a.nslot + slot) * 2 * D;
  for (int t = tid; t < 2 * D; t += 256) {
    const int which = t / D, e = t % D;
    svk[t] = sign * (((sRed[0][which][e] + sRed[1][which][e]) + sRed[2][which][e]) + sRed[3][which][e]);
  }
}

// ------------------------------------------------------------------------------------
// Stage 1: window-row statistics + candidate covariance, sums and value norms.
// ------------------------------------------------------------------------------------
template <class T, int D, int MTW>
__global__ void __launch_bounds__(256) k_rows_cov(CompressArgs a) {
  constexpr int KS = D / 32, DG = D / 8, PAD = 16 / (int)sizeof(T);
  constexpr int LDK = D + PAD, LDT = TILE + PAD;
  constexpr int CPT = TILE * DG / 256;   // 8-element chunks per thread per tensor
  constexpr int QM = CovSplit<D>::QM, QN = CovSplit<D>::QN;
  __shared__ __align__(16) T sK[TILE][LDK];
  __shared__ __align__(16) T sKT[D][LDT];
  __shared__ __align__(16) T sVT[D][LDT];
  __shared__ float sRed[4][2][D];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, sl = blockIdx.x;
  const T* Kh = reinterpret_cast<const T*>(a.k) + (size_t)head * a.N * D;
  const T* Vh = reinterpret_cast<const T*>(a.v) + (size_t)head * a.N * D;
  const int c_lo = a.n_s, c_hi = a.N - a.w;
  const int RT = (a.R + 15) >> 4;
  const float c2 = a.scale * kLog2e;

  typename Frag<T>::type qf[MTW][KS];
  int lim[MTW][4];     // last visible key position of each of the lane's rows (-1: padding)
  float rm[MTW][4], rl[MTW][4];
#pragma unroll
  for (int k = 0; k < MTW; ++k) {
    const int mt = wave + 4 * k;
    const int r = 16 * mt + (lane & 15);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[k][ks] = (mt < RT && r < a.R) ? load_frag(window_row<T>(a, head, r) + 32 * ks + 8 * (lane >> 4))
                                       : zero_frag<T>();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = 16 * mt + 4 * (lane >> 4) + i;
      lim[k][i] = (mt < RT && rr < a.R) ? a.N - a.w + rr % a.w : -1;
      rm[k][i] = -INFINITY;
      rl[k][i] = 0.f;
    }
  }
  f32x4 cacc[QM][QN];
#pragma unroll
  for (int mi = 0; mi < QM; ++mi)
#pragma unroll
    for (int ni = 0; ni < QN; ++ni) cacc[mi][ni] = zero4();
  float sk[8], sv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) sk[e] = sv[e] = 0.f;
  const int dg = tid % DG;

  const int t_beg = sl * a.tps1, t_end = min(t_beg + a.tps1, a.ntile);
  for (int t = t_beg; t < t_end; ++t) {
    const int tok0 = t * TILE;
    const bool tile_has_cand = tok0 < c_hi && tok0 + TILE > c_lo;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + 256 * i;
      const int tt = c / DG;
      const int j = tok0 + tt;
      const bool cand = j >= c_lo && j < c_hi;
      typename Frag<T>::type kf = zero_frag<T>(), vf = zero_frag<T>();
      if (j < a.N) kf = load_frag(Kh + (size_t)j * D + 8 * dg);
      if (cand) vf = load_frag(Vh + (size_t)j * D + 8 * dg);
      store_frag(&sK[tt][8 * dg], kf);
      float ss = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sKT[8 * dg + e][tt] = cand ? raw_elem(kf, e) : raw_elem(zero_frag<T>(), e);
        sVT[8 * dg + e][tt] = raw_elem(vf, e);
        const float x = elem_f(vf, e);
        ss += x * x;
        sv[e] += x;
        sk[e] += cand ? elem_f(kf, e) : 0.f;
      }
      ss = row_group_sum<DG>(ss);
      if (cand && (lane % DG) == 0) a.vnorm[(size_t)head * a.n_c + (j - c_lo)] = sqrtf(ss);
    }
    __syncthreads();

    // window logits for this wave's row tiles; per-lane online (max, sum)
#pragma unroll
    for (int k = 0; k < MTW; ++k) {
      const int mt = wave + 4 * k;
      if (mt >= RT) continue;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          mma(acc, qf[k][ks], load_frag(&sK[16 * nt + (lane & 15)][32 * ks + 8 * (lane >> 4)]));
        const int j = tok0 + 16 * nt + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (j <= lim[k][i] && j < a.N) {
            const float s2 = acc[i] * c2;
            if (s2 > rm[k][i]) {
              rl[k][i] = rl[k][i] * fast_exp2(rm[k][i] - s2) + 1.f;
              rm[k][i] = s2;
            } else {
              rl[k][i] += fast_exp2(s2 - rm[k][i]);
            }
          }
        }
      }
    }
    if (tile_has_cand) cov_tile<T, D, LDT>(sVT, sKT, cacc, wave, lane);
    __syncthreads();
  }

  // merge the per-lane row statistics over the 16 lanes holding a row
#pragma unroll
  for (int k = 0; k < MTW; ++k)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float m = rm[k][i], l = rl[k][i];
      ml_merge(m, l, dpp_f<0x128>(m), dpp_f<0x128>(l));
      ml_merge(m, l, dpp_f<0x124>(m), dpp_f<0x124>(l));
      ml_merge(m, l, dpp_f<0x122>(m), dpp_f<0x122>(l));
      ml_merge(m, l, dpp_f<0x121>(m), dpp_f<0x121>(l));
      const int mt = wave + 4 * k;
      const int r = 16 * mt + 4 * (lane >> 4) + i;
      if ((lane & 15) == 0 && mt < RT && r < a.R) {
        float* rp = a.rowpart + (((size_t)head * a.nsl1 + sl) * a.R + r) * 2;
        rp[0] = m;
        rp[1] = l;
      }
    }
  write_cov_partials<T, D>(a, head, sl, cacc, sv, sk, 1.f, sRed, tid);
}

// ------------------------------------------------------------------------------------
// Stage 2: merge row partials -> (max, 1/Z) per window row.
// ------------------------------------------------------------------------------------
__global__ void __launch_bounds__(256) k_row_combine(CompressArgs a) {
  const int head = blockIdx.x;
  for (int r = threadIdx.x; r < a.R; r += blockDim.x) {
    float m = -INFINITY, l = 0.f;
    for (int s = 0; s < a.nsl1; ++s) {
      const float* rp = a.rowpart + (((size_t)head * a.nsl1 + s) * a.R + r) * 2;
      ml_merge(m, l, rp[0], rp[1]);
    }
    a.rowstat[((size_t)head * a.R + r) * 2 + 0] = m;
    a.rowstat[((size_t)head * a.R + r) * 2 + 1] = 1.f / l;
  }
}

// ------------------------------------------------------------------------------------
// Stage 3: window attention mass a_j, chunk pooling, provisional score.
// ------------------------------------------------------------------------------------
template <class T, int D, int MTW>
__global__ void __launch_bounds__(256) k_mass(CompressArgs a) {
  constexpr int KS = D / 32, DG = D / 8, PAD = 16 / (int)sizeof(T);
  constexpr int LDK = D + PAD;
  constexpr int CPT = TILE * DG / 256;
  __shared__ __align__(16) T sK[TILE][LDK];
  __shared__ float sA[4][TILE];
  __shared__ float sAj[TILE];
  __shared__ float sRow[512][2];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, sl = blockIdx.x;
  const T* Kh = reinterpret_cast<const T*>(a.k) + (size_t)head * a.N * D;
  const int c_lo = a.n_s, c_hi = a.N - a.w;
  const int RT = (a.R + 15) >> 4;
  const float c2 = a.scale * kLog2e;
  const float inv_rows = 1.f / (float)a.R;

  for (int r = tid; r < a.R; r += 256) {
    sRow[r][0] = a.rowstat[((size_t)head * a.R + r) * 2 + 0];
    sRow[r][1] = a.rowstat[((size_t)head * a.R + r) * 2 + 1];
  }
  typename Frag<T>::type qf[MTW][KS];
#pragma unroll
  for (int k = 0; k < MTW; ++k) {
    const int mt = wave + 4 * k;
    const int r = 16 * mt + (lane & 15);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[k][ks] = (mt < RT && r < a.R) ? load_frag(window_row<T>(a, head, r) + 32 * ks + 8 * (lane >> 4))
                                       : zero_frag<T>();
  }
  const int dg = tid % DG;
  __syncthreads();

  const int t_beg = sl * a.tps1, t_end = min(t_beg + a.tps1, a.ntile);
  for (int t = t_beg; t < t_end; ++t) {
    const int tok0 = t * TILE;
    if (!(tok0 < c_hi && tok0 + TILE > c_lo)) continue;  // uniform: no candidate here
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + 256 * i;
      const int tt = c / DG;
      const int j = tok0 + tt;
      typename Frag<T>::type kf = zero_frag<T>();
      if (j >= c_lo && j < c_hi) kf = load_frag(Kh + (size_t)j * D + 8 * dg);
      store_frag(&sK[tt][8 * dg], kf);
    }
    __syncthreads();
    float col[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < MTW; ++k) {
      const int mt = wave + 4 * k;
      if (mt >= RT) continue;
      float rmax[4], rinv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 16 * mt + 4 * (lane >> 4) + i;
        const bool ok = r < a.R;
        rmax[i] = ok ? sRow[r][0] : 0.f;
        rinv[i] = ok ? sRow[r][1] : 0.f;
      }
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          mma(acc, qf[k][ks], load_frag(&sK[16 * nt + (lane & 15)][32 * ks + 8 * (lane >> 4)]));
#pragma unroll
        for (int i = 0; i < 4; ++i) col[nt] += fast_exp2(acc[i] * c2 - rmax[i]) * rinv[i];
      }
    }
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const float x = cross_row_sum(col[nt]);
      if (lane < 16) sA[wave][16 * nt + lane] = x;
    }
    __syncthreads();
    if (tid < TILE) sAj[tid] = (((sA[0][tid] + sA[1][tid]) + sA[2][tid]) + sA[3][tid]) * inv_rows;
    __syncthreads();
    if (tid < TILE) {
      const int j = tok0 + tid;
      if (j >= c_lo && j < c_hi) {
        const int cs = (j / a.chunk) * a.chunk;
        const int lo = max(cs, c_lo), hi = min(cs + a.chunk, c_hi);
        float s = 0.f;
        for (int i = lo; i < hi; ++i) s += sAj[i - tok0];
        const float ab = s / (float)(hi - lo);
        const size_t o = (size_t)head * a.n_c + (j - c_lo);
        a.abar[o] = ab;
        a.score0[o] = ab * a.vnorm[o];
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------------------------
// Stage 4/9: per-head radix select of the k best scores (ties: lower position first),
// output in ascending position order.  Scores are non-negative floats, so their bit
// patterns order like unsigned integers.
// ------------------------------------------------------------------------------------
constexpr int TK_THREADS = 1024;
constexpr int TK_WAVES = TK_THREADS / 64;

__device__ __forceinline__ uint32_t score_key(float s) {
  uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? 0u : u;  // -0 and negatives sort as 0
}

// Exclusive block scan of one int per thread; returns the prefix, total in *total.
__device__ int block_excl_scan(int x, int* sW, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(inc, o);
    if (lane >= o) inc += y;
  }
  if (lane == 63) sW[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    int v = lane < TK_WAVES ? sW[lane] : 0;
    int vi = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int y = __shfl_up(vi, o);
      if (lane >= o) vi += y;
    }
    if (lane < TK_WAVES) sW[TK_WAVES + lane] = vi - v;  // exclusive wave offsets
    if (lane == TK_WAVES - 1) sW[2 * TK_WAVES] = vi;
  }
  __syncthreads();
  const int res = sW[TK_WAVES + wave] + inc - x;
  *total = sW[2 * TK_WAVES];
  __syncthreads();
  return res;
}

__global__ void __launch_bounds__(TK_THREADS) k_topk(const float* __restrict__ scores, int n,
                                                       int k, int32_t* __restrict__ out,
                                                       int out_stride, int pos_offset) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_prefix, sh_remaining;
  __shared__ int sW[2 * TK_WAVES + 1];
  const int tid = threadIdx.x, lane = tid & 63;
  const int head = blockIdx.x;
  const float* s = scores + (size_t)head * n;
  int32_t* o = out + (size_t)head * out_stride;
  if (k <= 0) return;

  uint32_t prefix = 0, mask = 0, remaining = (uint32_t)k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = tid; i < 256; i += TK_THREADS) hist[i] = 0;
    __syncthreads();
    for (int base = 0; base < n; base += TK_THREADS) {
      const int j = base + tid;
      uint32_t u = 0;
      bool active = false;
      if (j < n) {
        u = score_key(s[j]);
        active = (u & mask) == prefix;
      }
      const uint32_t d = (u >> shift) & 255u;
      // aggregate equal digits within the wave (scores tend to share high bits)
      unsigned long long act = __ballot(active);
      for (int it = 0; it < 4 && act; ++it) {
        const int leader = __ffsll((long long)act) - 1;
        const uint32_t dl = __shfl(d, leader);
        const unsigned long long same = __ballot(active && d == dl);
        if (lane == leader) atomicAdd(&hist[dl], (uint32_t)__popcll(same));
        if (active && d == dl) active = false;
        act &= ~same;
      }
      if (active) atomicAdd(&hist[d], 1u);
    }
    __syncthreads();
    if (tid == 0) {
      uint32_t cum = 0;
      int chosen = 0;
      for (int bin = 255; bin >= 0; --bin) {
        if (cum + hist[bin] >= remaining) { chosen = bin; break; }
        cum += hist[bin];
      }
      sh_prefix = prefix | ((uint32_t)chosen << shift);
      sh_remaining = remaining - cum;
    }
    __syncthreads();
    prefix = sh_prefix;
    remaining = sh_remaining;
    mask |= 255u << shift;
    __syncthreads();
  }
  // keys > T are all kept; of the keys == T the `need` lowest positions are kept
  const uint32_t T = prefix;
  const int need = (int)remaining;
  constexpr int IT = 4;
  int eq_carry = 0, out_carry = 0;
  for (int base = 0; base < n; base += TK_THREADS * IT) {
    uint32_t u[IT];
    int n_eq = 0;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int j = base + tid * IT + it;
      u[it] = j < n ? score_key(s[j]) : 0u;
      n_eq += (j < n && u[it] == T);
    }
    int eq_tot;
    int eq_before = block_excl_scan(n_eq, sW, &eq_tot) + eq_carry;
    bool take[IT];
    int n_take = 0;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int j = base + tid * IT + it;
      bool tk = false;
      if (j < n) {
        if (u[it] > T) tk = true;
        else if (u[it] == T) { tk = eq_before < need; ++eq_before; }
      }
      take[it] = tk;
      n_take += tk;
    }
    int out_tot;
    int pos = block_excl_scan(n_take, sW, &out_tot) + out_carry;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      if (take[it]) {
        if (pos < k) o[pos] = base + tid * IT + it + pos_offset;
        ++pos;
      }
    }
    eq_carry += eq_tot;
    out_carry += out_tot;
  }
}

// ------------------------------------------------------------------------------------
// Stage 5: rows of the provisional kept set -> compact buffer [H, kmax, D].
// ------------------------------------------------------------------------------------
template <class T, int D>
__global__ void __launch_bounds__(256) k_gather_rows(CompressArgs a) {
  constexpr int DG = D / 8;
  const int head = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int i = c / DG, dg = c % DG;
  if (i >= a.k_keep) return;
  const int pos = a.kept0[(size_t)head * a.kmax + i];
  const size_t src = ((size_t)head * a.N + pos) * D + 8 * dg;
  const size_t dst = ((size_t)head * a.kmax + i) * D + 8 * dg;
  store_frag(reinterpret_cast<T*>(a.gath_k) + dst, load_frag(reinterpret_cast<const T*>(a.k) + src));
  store_frag(reinterpret_cast<T*>(a.gath_v) + dst, load_frag(reinterpret_cast<const T*>(a.v) + src));
}

// ------------------------------------------------------------------------------------
// Stage 6/11: covariance and sums of `nrows` consecutive rows, stored negated into the
// slots after the candidate slices.
// ------------------------------------------------------------------------------------
template <class T, int D>
__global__ void __launch_bounds__(256) k_cov_rows(CompressArgs a, const void* kbase,
                                                   const void* vbase, int head_rows,
                                                   int row_off, int nrows) {
  constexpr int DG = D / 8, PAD = 16 / (int)sizeof(T);
  constexpr int LDT = TILE + PAD;
  constexpr int CPT = TILE * DG / 256;
  constexpr int QM = CovSplit<D>::QM, QN = CovSplit<D>::QN;
  __shared__ __align__(16) T sKT[D][LDT];
  __shared__ __align__(16) T sVT[D][LDT];
  __shared__ float sRed[4][2][D];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, sl = blockIdx.x;
  const T* Kh = reinterpret_cast<const T*>(kbase) + ((size_t)head * head_rows + row_off) * D;
  const T* Vh = reinterpret_cast<const T*>(vbase) + ((size_t)head * head_rows + row_off) * D;
  f32x4 cacc[QM][QN];
#pragma unroll
  for (int mi = 0; mi < QM; ++mi)
#pragma unroll
    for (int ni = 0; ni < QN; ++ni) cacc[mi][ni] = zero4();
  float sk[8], sv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) sk[e] = sv[e] = 0.f;
  const int dg = tid % DG;
  const int ntiles = (nrows + TILE - 1) / TILE;
  const int t_beg = sl * a.tpsr, t_end = min(t_beg + a.tpsr, ntiles);
  for (int t = t_beg; t < t_end; ++t) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + 256 * i;
      const int tt = c / DG;
      const int j = t * TILE + tt;
      typename Frag<T>::type kf = zero_frag<T>(), vf = zero_frag<T>();
      if (j < nrows) {
        kf = load_frag(Kh + (size_t)j * D + 8 * dg);
        vf = load_frag(Vh + (size_t)j * D + 8 * dg);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sKT[8 * dg + e][tt] = raw_elem(kf, e);
        sVT[8 * dg + e][tt] = raw_elem(vf, e);
        sv[e] += elem_f(vf, e);
        sk[e] += elem_f(kf, e);
      }
    }
    __syncthreads();
    cov_tile<T, D, LDT>(sVT, sKT, cacc, wave, lane);
    __syncthreads();
  }
  write_cov_partials<T, D>(a, head, a.nsl1 + sl, cacc, sv, sk, -1.f, sRed, tid);
}

// ------------------------------------------------------------------------------------
// Stage 7/12: fixed-order sum of the slots.  final == 0: centre, clamp and keep the
// provisional summary; final == 1: write the raw output moments.
// ------------------------------------------------------------------------------------
template <int D, bool BF16>
__global__ void __launch_bounds__(256) k_reduce(CompressArgs a, int final_pass) {
  __shared__ float sTot[2][D];
  const int tid = threadIdx.x;
  const int head = blockIdx.y;
  const int n = a.n_c - a.k_keep;  // evicted count
  for (int t = tid; t < 2 * D; t += 256) {
    float acc = 0.f;
    for (int s = 0; s < a.nslot; ++s) acc += a.svkpart[((size_t)head * a.nslot + s) * 2 * D + t];
    sTot[t / D][t % D] = acc;  // [0] = s_v, [1] = s_k
  }
  __syncthreads();
  const int e0 = (blockIdx.x * 256 + tid) * 4;
  if (e0 < D * D) {
    const int row = e0 / D, col = e0 % D;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < a.nslot; ++s) {
      const float4 p = *reinterpret_cast<const float4*>(a.spart + ((size_t)head * a.nslot + s) * D * D + e0);
      acc.x += p.x; acc.y += p.y; acc.z += p.z; acc.w += p.w;
    }
    if (final_pass) {
      *reinterpret_cast<float4*>(a.S + (size_t)head * D * D + e0) = acc;
    } else {
      const float inv_n = 1.f / (float)n;
      const float sv = sTot[0][row];
      float st[4] = {acc.x - sv * sTot[1][col] * inv_n, acc.y - sv * sTot[1][col + 1] * inv_n,
                     acc.z - sv * sTot[1][col + 2] * inv_n, acc.w - sv * sTot[1][col + 3] * inv_n};
#pragma unroll
      for (int i = 0; i < 4; ++i) if (fabsf(st[i]) < a.tau) st[i] = 0.f;
      *reinterpret_cast<float4*>(a.stil + (size_t)head * D * D + e0) = make_float4(st[0], st[1], st[2], st[3]);
      if (BF16) {
        bf16_t* hl = reinterpret_cast<bf16_t*>(a.stil_hl) + (size_t)head * 2 * D * D;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bf16_t hi = f2bf(st[i]);
          hl[e0 + i] = hi;
          hl[D * D + e0 + i] = f2bf(st[i] - bf2f(hi));
        }
      }
    }
  }
  if (blockIdx.x == 0) {
    if (final_pass) {
      for (int t = tid; t < D; t += 256) {
        a.s_v[(size_t)head * D + t] = sTot[0][t];
        a.s_k[(size_t)head * D + t] = sTot[1][t];
      }
      if (tid == 0) a.n_e[head] = n;
    } else {
      for (int t = tid; t < D; t += 256) a.vbar[(size_t)head * D + t] = sTot[0][t] / (float)n;
    }
  }
}

// ------------------------------------------------------------------------------------
// Stage 8: moment residual score of every candidate.
// ------------------------------------------------------------------------------------
template <class T, int D>
__global__ void __launch_bounds__(256) k_residual(CompressArgs a) {
  constexpr int KS = D / 32, PAD = 16 / (int)sizeof(T);
  constexpr int LDS_ = D + PAD;
  constexpr bool BF = sizeof(T) == 2;
  constexpr int NPL = BF ? 2 : 1;  // planes: bf16 hi + lo, or fp32
  __shared__ __align__(16) T sS[NPL][D][LDS_];
  __shared__ float sVbar[D];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, sl = blockIdx.x;
  const int c_lo = a.n_s, c_hi = a.N - a.w;
  const float coef = a.scale / (float)(a.n_c - a.k_keep);
  const T* Kh = reinterpret_cast<const T*>(a.k) + (size_t)head * a.N * D;
  const T* Vh = reinterpret_cast<const T*>(a.v) + (size_t)head * a.N * D;
  {
    const T* src = BF ? reinterpret_cast<const T*>(a.stil_hl) + (size_t)head * 2 * D * D
                      : reinterpret_cast<const T*>(a.stil) + (size_t)head * D * D;
    for (int c = tid; c < NPL * D * D / 8; c += 256) {
      const int pl = c / (D * D / 8), rem = c % (D * D / 8);
      const int row = rem / (D / 8), cg = rem % (D / 8);
      store_frag(&sS[pl][row][8 * cg], load_frag(src + (size_t)pl * D * D + (size_t)row * D + 8 * cg));
    }
    for (int t = tid; t < D; t += 256) sVbar[t] = a.vbar[(size_t)head * D + t];
  }
  __syncthreads();

  for (int it = 0; it < a.tps3; ++it) {
    const int base = c_lo + ((sl * a.tps3 + it) * 4 + wave) * TILE;
    if (base >= c_hi) break;
    typename Frag<T>::type kf[4][KS];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const int j = base + 16 * nt + (lane & 15);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kf[nt][ks] = j < c_hi ? load_frag(Kh + (size_t)j * D + 32 * ks + 8 * (lane >> 4)) : zero_frag<T>();
    }
    float rho[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
    for (int mt = 0; mt < D / 16; ++mt) {
      f32x4 acc[4];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) acc[nt] = zero4();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
        for (int pl = 0; pl < NPL; ++pl) {
          const typename Frag<T>::type af = load_frag(&sS[pl][16 * mt + (lane & 15)][32 * ks + 8 * (lane >> 4)]);
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) mma(acc[nt], af, kf[nt][ks]);
        }
      }
      const int a0 = 16 * mt + 4 * (lane >> 4);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int j = base + 16 * nt + (lane & 15);
        if (j < c_hi) {
          float v[4];
          load4(Vh + (size_t)j * D + a0, v);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float r = v[i] - sVbar[a0 + i] - coef * acc[nt][i];
            rho[nt] += r * r;
          }
        }
      }
    }
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const float x = cross_row_sum(rho[nt]);
      const int j = base + 16 * nt + (lane & 15);
      if (lane < 16 && j < c_hi) {
        const size_t o = (size_t)head * a.n_c + (j - c_lo);
        a.score[o] = a.abar[o] * sqrtf(x);
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// Stage 10: retained rows (sinks, kept candidates, window) -> k_out/v_out, idx, lens.
// With budget >= N every row is retained.
// ------------------------------------------------------------------------------------
template <class T, int D>
__global__ void __launch_bounds__(256) k_gather_out(CompressArgs a, int n_out, int keep_all) {
  constexpr int DG = D / 8;
  const int head = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int i = c / DG, dg = c % DG;
  if (blockIdx.x == 0 && threadIdx.x == 0) a.lens_out[head] = n_out;
  if (i >= n_out) return;
  int pos;
  if (keep_all || i < a.n_s) pos = i;
  else if (i < a.n_s + a.k_keep) pos = a.kept[(size_t)head * a.kmax + (i - a.n_s)];
  else pos = a.N - a.w + (i - a.n_s - a.k_keep);
  const size_t src = ((size_t)head * a.N + pos) * D + 8 * dg;
  const size_t dst = ((size_t)head * a.cap + i) * D + 8 * dg;
  store_frag(reinterpret_cast<T*>(a.k_out) + dst, load_frag(reinterpret_cast<const T*>(a.k) + src));
  store_frag(reinterpret_cast<T*>(a.v_out) + dst, load_frag(reinterpret_cast<const T*>(a.v) + src));
  if (dg == 0) a.idx_out[(size_t)head * n_out + i] = pos;
}

template <int D>
__global__ void __launch_bounds__(256) k_zero_moments(CompressArgs a) {
  const int head = blockIdx.y;
  for (int e = blockIdx.x * 256 + threadIdx.x; e < D * D; e += gridDim.x * 256)
    a.S[(size_t)head * D * D + e] = 0.f;
  if (blockIdx.x == 0) {
    for (int t = threadIdx.x; t < D; t += 256) {
      a.s_k[(size_t)head * D + t] = 0.f;
      a.s_v[(size_t)head * D + t] = 0.f;
    }
    if (threadIdx.x == 0) a.n_e[head] = 0;
  }
}

// ------------------------------------------------------------------------------------
#define MKV_CHECK_LAUNCH()                  \
  do {                                      \
    hipError_t e_ = hipGetLastError();      \
    if (e_ != hipSuccess) return e_;        \
  } while (0)

template <class T, int D, int MTW>
static hipError_t run_compress(const CompressArgs& a, hipStream_t st, float* dbg_abar,
                               float* dbg_score0, float* dbg_score, int32_t* dbg_kept0) {
  constexpr bool BF = sizeof(T) == 2;
  const dim3 blk(256);
  const int H = a.H;
  if (a.L >= a.N) {
    const int n_out = a.N;
    hipLaunchKernelGGL((k_gather_out<T, D>), dim3((n_out * (D / 8) + 255) / 256, H), blk, 0, st, a, n_out, 1);
    MKV_CHECK_LAUNCH();
    hipLaunchKernelGGL((k_zero_moments<D>), dim3(4, H), blk, 0, st, a);
    MKV_CHECK_LAUNCH();
    return hipSuccess;
  }
  hipLaunchKernelGGL((k_rows_cov<T, D, MTW>), dim3(a.nsl1, H), blk, 0, st, a);
  MKV_CHECK_LAUNCH();
  hipLaunchKernelGGL(k_row_combine, dim3(H), blk, 0, st, a);
  MKV_CHECK_LAUNCH();
  hipLaunchKernelGGL((k_mass<T, D, MTW>), dim3(a.nsl1, H), blk, 0, st, a);
  MKV_CHECK_LAUNCH();
  const float* first_scores = a.mi_rounds < 0 ? a.abar : a.score0;
  int32_t* first_out = a.mi_rounds >= 1 ? a.kept0 : a.kept;
  hipLaunchKernelGGL(k_topk, dim3(H), dim3(TK_THREADS), 0, st, first_scores, a.n_c, a.k_keep,
                     first_out, a.kmax, a.n_s);
  MKV_CHECK_LAUNCH();
  const dim3 red_grid((D * D / 4 + 255) / 256, H);
  if (a.mi_rounds >= 1) {
    if (a.k_keep > 0) {
      hipLaunchKernelGGL((k_gather_rows<T, D>), dim3((a.k_keep * (D / 8) + 255) / 256, H), blk, 0, st, a);
      MKV_CHECK_LAUNCH();
      hipLaunchKernelGGL((k_cov_rows<T, D>), dim3(a.nslr, H), blk, 0, st, a, (const void*)a.gath_k,
                         (const void*)a.gath_v, a.kmax, 0, a.k_keep);
      MKV_CHECK_LAUNCH();
    }
    hipLaunchKernelGGL((k_reduce<D, BF>), red_grid, blk, 0, st, a, 0);
    MKV_CHECK_LAUNCH();
    hipLaunchKernelGGL((k_residual<T, D>), dim3(a.nsl3, H), blk, 0, st, a);
    MKV_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_topk, dim3(H), dim3(TK_THREADS), 0, st, (const float*)a.score, a.n_c,
                       a.k_keep, a.kept, a.kmax, a.n_s);
    MKV_CHECK_LAUNCH();
  }
  hipLaunchKernelGGL((k_gather_out<T, D>), dim3((a.L * (D / 8) + 255) / 256, H), blk, 0, st, a, a.L, 0);
  MKV_CHECK_LAUNCH();
  if (a.k_keep > 0) {
    hipLaunchKernelGGL((k_cov_rows<T, D>), dim3(a.nslr, H), blk, 0, st, a, (const void*)a.k_out,
                       (const void*)a.v_out, a.cap, a.n_s, a.k_keep);
    MKV_CHECK_LAUNCH();
  }
  hipLaunchKernelGGL((k_reduce<D, BF>), red_grid, blk, 0, st, a, 1);
  MKV_CHECK_LAUNCH();
  // diagnostics
  const size_t nc_bytes = (size_t)H * a.n_c * sizeof(float);
  if (dbg_abar && hipMemcpyAsync(dbg_abar, a.abar, nc_bytes, hipMemcpyDeviceToDevice, st) != hipSuccess)
    return hipGetLastError();
  if (dbg_score0 && a.mi_rounds >= 0 &&
      hipMemcpyAsync(dbg_score0, a.score0, nc_bytes, hipMemcpyDeviceToDevice, st) != hipSuccess)
    return hipGetLastError();
  if (dbg_score && a.mi_rounds >= 1 &&
      hipMemcpyAsync(dbg_score, a.score, nc_bytes, hipMemcpyDeviceToDevice, st) != hipSuccess)
    return hipGetLastError();
  if (dbg_kept0 && a.k_keep > 0) {
    const int32_t* src = a.mi_rounds >= 1 ? a.kept0 : a.kept;
    if (hipMemcpy2DAsync(dbg_kept0, (size_t)a.k_keep * 4, src, (size_t)a.kmax * 4, (size_t)a.k_keep * 4,
                         H, hipMemcpyDeviceToDevice, st) != hipSuccess)
      return hipGetLastError();
  }
  return hipSuccess;
}

template <class T, int D>
static hipError_t run_compress_r(const CompressArgs& a, hipStream_t st, float* d0, float* d1,
                                 float* d2, int32_t* d3) {
  const int rt = (a.R + 15) / 16;         // 16-row tiles of window queries
  const int mtw = (rt + 3) / 4;           // tiles per wave
  if (mtw <= 2) return run_compress<T, D, 2>(a, st, d0, d1, d2, d3);
  if (mtw <= 4) return run_compress<T, D, 4>(a, st, d0, d1, d2, d3);
  return run_compress<T, D, 8>(a, st, d0, d1, d2, d3);
}

hipError_t launch_compress(const CompressArgs& a, bool bf16, hipStream_t st, float* dbg_abar,
                           float* dbg_score0, float* dbg_score, int32_t* dbg_kept0) {
  if (bf16)
    return a.D == 64 ? run_compress_r<bf16_t, 64>(a, st, dbg_abar, dbg_score0, dbg_score, dbg_kept0)
                     : run_compress_r<bf16_t, 128>(a, st, dbg_abar, dbg_score0, dbg_score, dbg_kept0);
  return a.D == 64 ? run_compress_r<float, 64>(a, st, dbg_abar, dbg_score0, dbg_score, dbg_kept0)
                   : run_compress_r<float, 128>(a, st, dbg_abar, dbg_score0, dbg_score, dbg_kept0);
}

}  // namespace mkv
