// One-shot prefill compression with moment-informed selection (Sec. 5.1 prefill
// protocol; Sec. 4.2 Eq. residual; App. A.1 Eqs. app_sufficient, app_S_tilde).
//
// Stages, all on the caller's stream (H = B*Hkv heads, C = [n_s, N-w) candidates):
//   1 k_rows_cov      per (slice of 64-token tiles, head): window logits Q.K^T on MFMA,
//                     per-row online (max, sum) over the visible keys; for candidate
//                     tokens also the covariance V^T K on MFMA (bf16: both operands
//                     read transposed out of the row-major LDS tiles, two tile buffers;
//                     fp32: tiles written transposed), the sums s_k, s_v and ||v_j||,
//                     one partial slot per slice.                         [reads K, V]
//   2 k_row_combine   per head: merge the row partials in slice order -> (max, 1/Z);
//                     add up the slices' slots into slot 0 (the candidates' sums);
//                     zero the head's two top-k key histograms.
//   3 k_mass          per (slice, head): logits again, softmax mass summed over the
//                     window rows -> a_j, aligned chunk pooling -> abar_j,
//                     provisional score abar_j ||v_j||, added to the key histogram of
//                     the first selection.                                 [reads K]
//   4 k_tk_*          per head: radix select of the k_keep best scores, lower position
//                     first on ties; writes the kept positions in ascending order; each
//                     slice's workgroup
//                     then adds the covariance and sums of its kept rows (read through
//                     their positions), stored negated as a partial slot, or, when the
//                     head's evicted rows are fewer than its kept ones, of its evicted
//                     rows, stored as they are.
//   7 k_reduce        fixed-order sum of the slots = raw moments of the provisional
//                     evicted set: slot 0 and the kept rows' slots (the candidates' sums
//                     minus the kept rows'), or only the evicted rows' slots.  Summing the evicted rows directly
//                     when they are the fewer keeps the cancellation of S_C - S_kept from
//                     growing with the ratio of candidates to evicted rows.
//   8 k_residual      per (slice, head): centring and clamp of the provisional summary
//                     into LDS (fp32, or a bf16 hi/lo pair), S_tilde k_j on MFMA,
//                     ||v_j - v_bar - c S_tilde k_j||, score_j = abar_j * that norm,
//                     added to the final selection's key histogram.       [reads K, V]
//   9 k_tk_*          kept set of the moment round and its covariance slots.
//                     mi_rounds > 1 repeats stages 7-9, each round scoring with the
//                     moments of the round before (k_reduce also clears the histogram
//                     the next k_residual fills).
//  10 k_finish        one launch: retained rows (sinks, kept, window) -> k_out/v_out,
//                     idx, lens; and the final raw moments S, s_k, s_v, n_e (the slots of
//                     the final selection's covariance, as in stage 7).
// Every reduction has a fixed order, so results are bit-reproducible.
#include "mkv_bf16.h"
#include "mkv_device.h"
#include "mkv_compress.h"

namespace mkv {

constexpr int TILE = 64;  // tokens per tile

// Top-k selection (lowest score evicted first): scores as monotone 32-bit keys, a
// per-head histogram of key bits 30..20 filled by the kernel that produces the scores,
// then slices of TKS positions.
constexpr int TKS = 2048;          // positions per slice
constexpr int TKT = 256;           // threads per slice workgroup
constexpr int TKPT = TKS / TKT;    // consecutive positions per thread
constexpr int TK_MAX_SLICES = 512; // 1048576 candidates
constexpr int TK_CAND_LDS = 8192;  // candidates of the k-th key's bin staged in LDS

__device__ __forceinline__ uint32_t score_key(float s) {
  uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? 0u : u;  // -0 and negatives sort as 0
}

constexpr int TK_HBINS = 2048;     // bins of the per-head histogram (key bits 30..20)

// Candidates kept by a head: the uniform k_keep, or its head-adaptive share (clamped to
// the buffers, since it sizes reads and writes).
__device__ __forceinline__ int head_keep(const CompressArgs& a, int head) {
  return a.kh ? min(max(a.kh[head], 0), a.kmax) : a.k_keep;
}

// A head whose evicted candidates are fewer than its kept ones gets its moments summed
// over the evicted rows; the others as the candidates' sums minus the kept rows'.
__device__ __forceinline__ bool direct_sums(const CompressArgs& a, int head) {
  const int k = head_keep(a, head);
  return a.n_c - k < k;
}

// Adds a workgroup's LDS histogram to the head's histogram in global memory (integer
// atomics: the result is exact whatever the order).
template <int NT>
__device__ __forceinline__ void hist_flush(const uint32_t* lh, uint32_t* gh) {
  for (int b = threadIdx.x; b < TK_HBINS; b += NT)
    if (lh[b]) atomicAdd(&gh[b], lh[b]);
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

// Covariance work split over the NW waves of a workgroup, in 16x16 MFMA tiles of the
// D x D output: wave w owns QM x QN tiles at rows a0(w), columns b0(w).
//   D=128: 4 waves -> 64x64 quadrants; 8 waves -> 32x64 blocks.
//   D=64:  4 waves -> 16x64 strips;    8 waves -> 16x32 blocks.
template <int D, int NW> struct CovSplit {
  static constexpr int QM = D == 128 ? (NW == 4 ? 4 : 2) : 1;
  static constexpr int QN = D == 128 ? 4 : (NW == 4 ? 4 : 2);
  static __device__ __forceinline__ int a0(int wave) {
    return D == 128 ? (NW == 4 ? 64 * (wave >> 1) : 32 * (wave >> 1)) : (NW == 4 ? 16 * wave : 16 * (wave >> 1));
  }
  static __device__ __forceinline__ int b0(int wave) {
    return D == 128 ? 64 * (wave & 1) : (NW == 4 ? 0 : 32 * (wave & 1));
  }
};

// Transposed tiles in LDS ([dim][token], rows padded by 16 bytes): for bf16 the 16-byte
// chunks of a row are XOR-swizzled by bits 3..5 of the row, so that the pair writes of a
// wave (16 column groups, i.e. rows 8g + c, one chunk) spread over the banks while every
// MFMA fragment read still fetches one whole chunk.  fp32 tiles are not swizzled.
template <class T>
__device__ __forceinline__ int tcol(int row, int col) {
  if constexpr (sizeof(T) == 2) return col ^ (((row >> 3) & 7) << 3);
  else return col;
}

// cacc += V_tile^T K_tile over the TILE tokens held transposed in LDS (fp32 tiles).
template <class T, int D, int NW, int LD>
__device__ __forceinline__ void cov_tile(const T (*sVT)[LD], const T (*sKT)[LD],
                                         f32x4 (&cacc)[CovSplit<D, NW>::QM][CovSplit<D, NW>::QN],
                                         int wave, int lane) {
  constexpr int QM = CovSplit<D, NW>::QM, QN = CovSplit<D, NW>::QN;
  const int a0 = CovSplit<D, NW>::a0(wave), b0 = CovSplit<D, NW>::b0(wave);
#pragma unroll
  for (int kk = 0; kk < TILE / 32; ++kk) {
    const int col = 32 * kk + 8 * (lane >> 4);
    typename Frag<T>::type af[QM];
#pragma unroll
    for (int mi = 0; mi < QM; ++mi) {
      const int r = a0 + 16 * mi + (lane & 15);
      af[mi] = load_frag(&sVT[r][tcol<T>(r, col)]);
    }
#pragma unroll
    for (int ni = 0; ni < QN; ++ni) {
      const int r = b0 + 16 * ni + (lane & 15);
      typename Frag<T>::type bf = load_frag(&sKT[r][tcol<T>(r, col)]);
#pragma unroll
      for (int mi = 0; mi < QM; ++mi) mma(cacc[mi][ni], af[mi], bf);
    }
  }
}

// The same from the tiles as they are (bf16, [token][dim], row stride ld): both operands
// read transposed out of LDS, so nothing is written transposed.
template <int D, int NW>
__device__ __forceinline__ void cov_tile_tr(const bf16_t* sV, const bf16_t* sK, int ld,
                                            f32x4 (&cacc)[CovSplit<D, NW>::QM][CovSplit<D, NW>::QN],
                                            int wave, int lane) {
  constexpr int QM = CovSplit<D, NW>::QM, QN = CovSplit<D, NW>::QN;
  const int a0 = CovSplit<D, NW>::a0(wave), b0 = CovSplit<D, NW>::b0(wave);
#pragma unroll
  for (int kk = 0; kk < TILE / 32; ++kk) {
    bf16x8 af[QM];
#pragma unroll
    for (int mi = 0; mi < QM; ++mi) af[mi] = lds_frag_tr(sV, ld, 32 * kk, a0 + 16 * mi, lane);
#pragma unroll
    for (int ni = 0; ni < QN; ++ni) {
      const bf16x8 bf = lds_frag_tr(sK, ld, 32 * kk, b0 + 16 * ni, lane);
#pragma unroll
      for (int mi = 0; mi < QM; ++mi) mma(cacc[mi][ni], af[mi], bf);
    }
  }
}

// Register staging of one 64-token tile of K and V for NT threads.  Thread t holds the
// 8-column group g = t % (D/8) of NP token pairs (2p, 2p+1), p = t / (D/8) + PSTEP * i:
// the lanes of a wave read whole rows (one load instruction covers 64 / (D/8) / 2 rows,
// contiguous 16-byte pieces); the rows go to LDS as they are (bf16) or transposed, as
// packed pairs of consecutive tokens (fp32).  With more threads than pieces of a tile (NT = 512, D = 64) the
// surplus threads hold nothing.
template <class T, int D, int NT> struct TileRegs {
  static constexpr int GROUPS = D / 8;
  static constexpr int PSTEP = NT / GROUPS;              // pairs covered by one register set
  static constexpr int NP = PSTEP >= TILE / 2 ? 1 : TILE / 2 / PSTEP;
  typename Frag<T>::type k[NP][2], v[NP][2];
  // Marks the point where the tile is used: the registers become opaque values there, so
  // no select or other use is moved up to the load (which would wait for it at once).
  __device__ __forceinline__ void arrive() {
#pragma unroll
    for (int i = 0; i < NP; ++i)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        asm volatile("" : "+v"(k[i][h]));
        asm volatile("" : "+v"(v[i][h]));
      }
  }
  static __device__ __forceinline__ bool active(int tid) { return tid < TILE / 2 * GROUPS; }
  static __device__ __forceinline__ int group(int tid) { return tid % GROUPS; }
  static __device__ __forceinline__ int pair(int tid, int i) {
    return min(tid / GROUPS, TILE / 2 - 1) + PSTEP * i;  // surplus threads: a valid pair
  }
};

__device__ __forceinline__ void store_pair(bf16_t* p, bf16_t lo, bf16_t hi) {
  *reinterpret_cast<uint32_t*>(p) = (uint32_t)lo | ((uint32_t)hi << 16);
}
__device__ __forceinline__ void store_pair(float* p, float lo, float hi) {
  *reinterpret_cast<float2*>(p) = make_float2(lo, hi);
}

// Rows row0 + 2p and row0 + 2p + 1 of K and V (head base pointers), clamped to the
// n_rows readable rows.  Every lane issues all of its loads and nothing selects on them
// here: a load under a per-lane branch, or a use right after it, would make the compiler
// wait for the loads at once (the prefetched tile's included) instead of where the tile
// is used.  Rows past the end are dropped where the tile is used.
template <class T, int D, int NT>
__device__ __forceinline__ void tile_load(TileRegs<T, D, NT>& R, const T* Kh, const T* Vh, int row0,
                                          int n_rows, int tid) {
  typedef TileRegs<T, D, NT> TR;
  const int col = 8 * TR::group(tid);
#pragma unroll
  for (int i = 0; i < TR::NP; ++i) {
    const int p = TR::pair(tid, i);
    const size_t r0 = (size_t)min(row0 + 2 * p, n_rows - 1) * D;
    const size_t r1 = (size_t)min(row0 + 2 * p + 1, n_rows - 1) * D;
    R.k[i][0] = load_frag(Kh + r0 + col);
    R.k[i][1] = load_frag(Kh + r1 + col);
    R.v[i][0] = load_frag(Vh + r0 + col);
    R.v[i][1] = load_frag(Vh + r1 + col);
  }
}

// Transposed copies K^T, V^T of the tile (the fp32 path; a bf16 variant with the copies
// written as they are follows) with the rows of tokens outside the summed set
// zeroed (flag in(j) of token j), running sums of k and v over the thread's 8 columns,
// and ||v_j||^2 of the thread's tokens over its columns (ss[i][h], token 2p_i + h).
// bf16: the two tokens' elements are paired with one byte permute per column, and the
// sums and squares use the bf16 dot2 instruction (exact products, fp32 accumulation).
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b),
                                         c, false);
}

template <class T, int D, int NT, int LDT, class In>
__device__ __forceinline__ void tile_store_t(const TileRegs<T, D, NT>& R, T (*sKT)[LDT],
                                             T (*sVT)[LDT], int tok0, In in, float (&sk)[8],
                                             float (&sv)[8], float (&ss)[TileRegs<T, D, NT>::NP][2],
                                             int tid) {
  typedef TileRegs<T, D, NT> TR;
  const int row = 8 * TR::group(tid);
  const bool act = TR::active(tid);
#pragma unroll
  for (int i = 0; i < TR::NP; ++i) {
    const int p = TR::pair(tid, i);
    const bool c0 = act && in(tok0 + 2 * p), c1 = act && in(tok0 + 2 * p + 1);
    ss[i][0] = ss[i][1] = 0.f;
    if constexpr (sizeof(T) == 2) {
      constexpr uint32_t ONES = 0x3F803F80u;  // (1.0, 1.0) in bf16
      const u32x4 k0 = __builtin_bit_cast(u32x4, R.k[i][0]), k1 = __builtin_bit_cast(u32x4, R.k[i][1]);
      const u32x4 v0 = __builtin_bit_cast(u32x4, R.v[i][0]), v1 = __builtin_bit_cast(u32x4, R.v[i][1]);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t a0 = c0 ? k0[w] : 0u, a1 = c1 ? k1[w] : 0u;
        const uint32_t b0 = c0 ? v0[w] : 0u, b1 = c1 ? v1[w] : 0u;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint32_t sel = h ? 0x07060302u : 0x05040100u;  // (token 0, token 1) of column 2w+h
          const uint32_t kp = __builtin_amdgcn_perm(a1, a0, sel);
          const uint32_t vp = __builtin_amdgcn_perm(b1, b0, sel);
          const int r = row + 2 * w + h;
          if (act) {
            *reinterpret_cast<uint32_t*>(&sKT[r][tcol<T>(r, 2 * p)]) = kp;
            *reinterpret_cast<uint32_t*>(&sVT[r][tcol<T>(r, 2 * p)]) = vp;
          }
          sk[2 * w + h] = dot2_bf16(kp, ONES, sk[2 * w + h]);
          sv[2 * w + h] = dot2_bf16(vp, ONES, sv[2 * w + h]);
        }
        ss[i][0] = dot2_bf16(b0, b0, ss[i][0]);
        ss[i][1] = dot2_bf16(b1, b1, ss[i][1]);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float k0 = c0 ? elem_f(R.k[i][0], e) : 0.f, k1 = c1 ? elem_f(R.k[i][1], e) : 0.f;
        const float x0 = c0 ? elem_f(R.v[i][0], e) : 0.f, x1 = c1 ? elem_f(R.v[i][1], e) : 0.f;
        if (act) {
          store_pair(&sKT[row + e][tcol<T>(row + e, 2 * p)], k0, k1);
          store_pair(&sVT[row + e][tcol<T>(row + e, 2 * p)], x0, x1);
        }
        ss[i][0] += x0 * x0;
        ss[i][1] += x1 * x1;
        sv[e] += x0 + x1;
        sk[e] += k0 + k1;
      }
    }
  }
}

// bf16 tiles kept as they are: V rows into sV ([token][dim], row stride LDV) with the rows
// of tokens outside the summed set zeroed (K rows are stored by the caller as they are;
// zero V rows take those tokens out of V^T K), and the same sums and squares as above.
template <int D, int NT, int LDV, class In>
__device__ __forceinline__ void tile_sums_nat(const TileRegs<bf16_t, D, NT>& R, bf16_t (*sV)[LDV],
                                              int tok0, In in, float (&sk)[8], float (&sv)[8],
                                              float (&ss)[TileRegs<bf16_t, D, NT>::NP][2], int tid) {
  typedef TileRegs<bf16_t, D, NT> TR;
  constexpr uint32_t ONES = 0x3F803F80u;  // (1.0, 1.0) in bf16
  const bool act = TR::active(tid);
#pragma unroll
  for (int i = 0; i < TR::NP; ++i) {
    const int p = TR::pair(tid, i);
    const bool c0 = act && in(tok0 + 2 * p), c1 = act && in(tok0 + 2 * p + 1);
    ss[i][0] = ss[i][1] = 0.f;
    const u32x4 k0 = __builtin_bit_cast(u32x4, R.k[i][0]), k1 = __builtin_bit_cast(u32x4, R.k[i][1]);
    const u32x4 v0 = __builtin_bit_cast(u32x4, R.v[i][0]), v1 = __builtin_bit_cast(u32x4, R.v[i][1]);
    u32x4 m0, m1;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t a0 = c0 ? k0[w] : 0u, a1 = c1 ? k1[w] : 0u;
      const uint32_t b0 = c0 ? v0[w] : 0u, b1 = c1 ? v1[w] : 0u;
      m0[w] = b0;
      m1[w] = b1;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint32_t sel = h ? 0x07060302u : 0x05040100u;  // (token 0, token 1) of column 2w+h
        sk[2 * w + h] = dot2_bf16(__builtin_amdgcn_perm(a1, a0, sel), ONES, sk[2 * w + h]);
        sv[2 * w + h] = dot2_bf16(__builtin_amdgcn_perm(b1, b0, sel), ONES, sv[2 * w + h]);
      }
      ss[i][0] = dot2_bf16(b0, b0, ss[i][0]);
      ss[i][1] = dot2_bf16(b1, b1, ss[i][1]);
    }
    if (act) {
      *reinterpret_cast<u32x4*>(&sV[2 * p][8 * TR::group(tid)]) = m0;
      *reinterpret_cast<u32x4*>(&sV[2 * p + 1][8 * TR::group(tid)]) = m1;
    }
  }
}

// Write one slot of covariance and (s_v, s_k) partials; `sign` = -1 for downdates.  The
// column sums of the threads sharing a column group are added within each wave (lanes
// g, g + 16, ... for D = 128) and then over the waves in order through `red`
// (NW * 2 * D floats of LDS that are free to reuse).
template <class T, int D, int NT>
__device__ __forceinline__ void write_cov_partials(
    const CompressArgs& a, int head, int slot,
    f32x4 (&cacc)[CovSplit<D, NT / 64>::QM][CovSplit<D, NT / 64>::QN],
    float (&sv)[8], float (&sk)[8], float sign, float* red, int tid) {
  constexpr int NW = NT / 64;
  constexpr int QM = CovSplit<D, NW>::QM, QN = CovSplit<D, NW>::QN;
  typedef TileRegs<T, D, NT> TR;
  constexpr int G = TR::GROUPS;  // 16 or 8: lanes sharing a group are G apart
  const int lane = tid & 63, wave = tid >> 6;
  const int a0 = CovSplit<D, NW>::a0(wave), b0 = CovSplit<D, NW>::b0(wave);
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
    const float x = same_group_sum<G>(sv[e]), y = same_group_sum<G>(sk[e]);
    if (lane < G && TR::active(tid)) {
      red[(wave * 2 + 0) * D + 8 * lane + e] = x;
      red[(wave * 2 + 1) * D + 8 * lane + e] = y;
    }
  }
  __syncthreads();
  constexpr int NWA = (TILE / 2 * G + 63) / 64 < NW ? (TILE / 2 * G + 63) / 64 : NW;  // waves holding data
  float* svk = a.svkpart + ((size_t)head * a.nslot + slot) * 2 * D;
  for (int c = tid; c < 2 * D; c += NT) {
    const int part = c / D, col = c % D;
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < NWA; ++w) acc += red[(w * 2 + part) * D + col];
    svk[c] = sign * acc;
  }
}

// ------------------------------------------------------------------------------------
// Stage 1: window-row statistics + candidate covariance, sums and value norms.
// ------------------------------------------------------------------------------------
constexpr int RC_THREADS = 512;  // k_rows_cov workgroup: 8 waves

template <class T, int D, int MTW>
__global__ void __launch_bounds__(RC_THREADS) k_rows_cov(CompressArgs a) {
  constexpr int NT = RC_THREADS, NW = NT / 64;
  constexpr bool BF = sizeof(T) == 2;  // bf16: K and V tiles as they are (transposed reads)
  constexpr int KS = D / 32, PAD = 16 / (int)sizeof(T);
  constexpr int LDK = BF ? D + 16 : D + PAD, LDT = TILE + PAD;  // bf16 rows padded by 32 bytes
  constexpr int QM = CovSplit<D, NW>::QM, QN = CovSplit<D, NW>::QN;
  typedef TileRegs<T, D, NT> TR;
  // bf16: two buffers, so that tile t + 1 is stored while slower waves still read tile t
  // (one barrier per tile); fp32, and bf16 with four row tiles per wave (registers): one
  constexpr int NB = BF && MTW < 4 ? 2 : 1;
  __shared__ __align__(16) T sK[NB][TILE][LDK];
  __shared__ __align__(16) T sV[NB][BF ? TILE : 1][LDK];  // bf16: V rows, candidates only
  __shared__ __align__(16) T sKT[BF ? 1 : D][LDT];       // fp32: K^T, V^T
  __shared__ __align__(16) T sVT[BF ? 1 : D][LDT];
  __shared__ float sVnorm[kRowsMaxTiles * TILE];  // ||v_j|| of the slice, written at the end

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, sl = blockIdx.x;
  const T* Kh = reinterpret_cast<const T*>(a.k) + (size_t)head * a.N * D;
  const T* Vh = reinterpret_cast<const T*>(a.v) + (size_t)head * a.N * D;
  const int c_lo = a.n_s, c_hi = a.N - a.w;
  const int RT = (a.R + 15) >> 4;
  const float c2 = a.scale * kLog2e;

  // window query row tiles of this wave: mt = wave + NW*k
  typename Frag<T>::type qf[MTW][KS];
  int lim[MTW][4];     // last visible key position of each of the lane's rows (-1: padding)
  float rm[MTW][4], rl[MTW][4];
#pragma unroll
  for (int k = 0; k < MTW; ++k) {
    const int mt = wave + NW * k;
    const int r = 16 * mt + (lane & 15);
    // rows past R repeat row R-1: their statistics are never stored (no select on the
    // loaded value, which would wait for it before the tile loads are issued)
    const T* qrow = window_row<T>(a, head, min(r, a.R - 1));
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[k][ks] = load_frag(qrow + 32 * ks + 8 * (lane >> 4));
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
  auto is_cand = [&](int j) { return j >= c_lo && j < c_hi; };

  const int t_beg = sl * a.tps1, t_end = min(t_beg + a.tps1, a.ntile);
  // Two tiles in flight: tile t is staged in R[t & 1], and the load of tile t + 2 is issued
  // into the same registers as soon as tile t has been written to LDS.  Every step issues
  // its loads whether or not the tile exists (rows clamped to the slice's last row) and
  // the loop always runs both steps, so the count of loads in flight is the same on every
  // path and the compiler waits for exactly the tile being used.
  const int slice_rows = min(t_end * TILE, a.N);
  auto issue = [&](TR& R, int t) {
    tile_load<T, D, NT>(R, Kh, Vh, t * TILE, slice_rows, tid);
  };
  auto step = [&](TR& R, int t) {
    const int tok0 = t * TILE;
    const bool tile_has_cand = tok0 < c_hi && tok0 + TILE > c_lo;
    const bool live = t < t_end;  // uniform; a step past the slice only issues loads
    T (*cK)[LDK] = sK[t & (NB - 1)];
    T (*cV)[LDK] = sV[t & (NB - 1)];
    R.arrive();
    if (live) {
      if (TR::active(tid)) {
#pragma unroll
        for (int i = 0; i < TR::NP; ++i) {
          const int p = TR::pair(tid, i);  // rows past N: their logits are masked
          store_frag(&cK[2 * p][8 * TR::group(tid)], R.k[i][0]);
          store_frag(&cK[2 * p + 1][8 * TR::group(tid)], R.k[i][1]);
        }
      }
      float ss[TR::NP][2];
      if constexpr (BF)
        tile_sums_nat<D, NT, LDK>(R, cV, tok0, is_cand, sk, sv, ss, tid);
      else
        tile_store_t<T, D, NT, LDT>(R, sKT, sVT, tok0, is_cand, sk, sv, ss, tid);
      // ||v_j||: the GROUPS lanes holding token j's columns are adjacent.  No global
      // store inside the tile loop: a store among the loads in flight would make the
      // compiler wait for all of them; the norms wait in LDS.
#pragma unroll
      for (int i = 0; i < TR::NP; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const float x = row_group_sum<TR::GROUPS>(ss[i][h]);
          if (TR::active(tid) && TR::group(tid) == 0)
            sVnorm[(t - t_beg) * TILE + 2 * TR::pair(tid, i) + h] = sqrtf(x);
        }
    }
    issue(R, t + 2);
    if (!live) return;
    __syncthreads();

    // window logits for this wave's row tiles; per-lane online (max, sum), updated once
    // per row and tile.  Only tiles reaching past position N-w need the causal/tail mask.
    const bool need_mask = tok0 + TILE - 1 > a.N - a.w;
#pragma unroll
    for (int k = 0; k < MTW; ++k) {
      const int mt = wave + NW * k;
      if (mt >= RT) continue;
      f32x4 acc[4];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        acc[nt] = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          mma(acc[nt], qf[k][ks], load_frag(&cK[16 * nt + (lane & 15)][32 * ks + 8 * (lane >> 4)]));
      }
      if (!need_mask) {
        // every logit finite: the max is taken on the raw products (c2 > 0, so scaling
        // after the max is exact), the scale folds into the exponent's FMA, and the
        // rescale is skipped when no lane's max grew (it would multiply by exactly 1)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float am = fmaxf(fmaxf(acc[0][i], acc[1][i]), fmaxf(acc[2][i], acc[3][i]));
          const float mn = fmaxf(rm[k][i], am * c2);
          float l = rl[k][i];
          if (__any(mn > rm[k][i])) l *= fast_exp2(rm[k][i] - mn);
          rl[k][i] = l + ((fast_exp2(fmaf(acc[0][i], c2, -mn)) + fast_exp2(fmaf(acc[1][i], c2, -mn))) +
                          (fast_exp2(fmaf(acc[2][i], c2, -mn)) + fast_exp2(fmaf(acc[3][i], c2, -mn))));
          rm[k][i] = mn;
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float x[4];
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) {
            const int jj = tok0 + 16 * nt + (lane & 15);
            x[nt] = (jj <= lim[k][i] && jj < a.N) ? acc[nt][i] * c2 : -INFINITY;
          }
          // with no finite logit yet, shifting by 0 keeps (-inf, 0)
          const float mn = fmaxf(rm[k][i], fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
          const float ms = mn == -INFINITY ? 0.f : mn;
          rl[k][i] = rl[k][i] * fast_exp2(rm[k][i] - ms) +
                     ((fast_exp2(x[0] - ms) + fast_exp2(x[1] - ms)) +
                      (fast_exp2(x[2] - ms) + fast_exp2(x[3] - ms)));
          rm[k][i] = mn;
        }
      }
    }
    if (tile_has_cand) {
      if constexpr (BF)
        cov_tile_tr<D, NW>(&cV[0][0], &cK[0][0], LDK, cacc, wave, lane);
      else
        cov_tile<T, D, NW, LDT>(sVT, sKT, cacc, wave, lane);
    }
    if constexpr (NB == 1) __syncthreads();  // the single buffer is written again next step
  };
  TR R0, R1;
  issue(R0, t_beg);
  __builtin_amdgcn_sched_barrier(0);  // keep the issue order: tile t_beg's loads first
  issue(R1, t_beg + 1);
  for (int t = t_beg; t < t_end; t += 2) {
    step(R0, t);
    step(R1, t + 1);
  }

  if constexpr (NB == 2) __syncthreads();  // the last tile read before sV is reused below
  // ||v_j|| of the slice's candidates
  for (int x = tid; x < (t_end - t_beg) * TILE; x += NT) {
    const int j = t_beg * TILE + x;
    if (is_cand(j)) a.vnorm[(size_t)head * a.n_c + (j - c_lo)] = sVnorm[x];
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
      const int mt = wave + NW * k;
      const int r = 16 * mt + 4 * (lane >> 4) + i;
      if ((lane & 15) == 0 && mt < RT && r < a.R) {
        float* rp = a.rowpart + (((size_t)head * a.nsl1 + sl) * a.R + r) * 2;
        rp[0] = m;
        rp[1] = l;
      }
    }
  static_assert(sizeof(sV) + sizeof(sVT) >= NW * 2 * D * sizeof(float), "LDS for the column sums");
  write_cov_partials<T, D, NT>(a, head, sl, cacc, sv, sk, 1.f,
                               BF ? reinterpret_cast<float*>(&sV[0][0][0]) : reinterpret_cast<float*>(&sVT[0][0]), tid);
}

// ------------------------------------------------------------------------------------
// Stage 2: merge row partials -> (max, 1/Z) per window row.  Eight lanes per row, each
// merging every eighth slice, then a fixed xor tree across the eight.  The same launch
// adds up the nsl1 candidate covariance slots of the head into slot 0 (same lane scheme:
// eight lanes per float4, each summing every eighth slot), so that the later sums of the
// moments read one slot for the candidates.  Each float4 is read and then written by the
// same eight lanes, so no other workgroup reads what slot 0 receives.
// ------------------------------------------------------------------------------------
template <int D> constexpr int reduce_blocks() { return ((D * D + 2 * D) / 4 + 31) / 32; }

template <int D>
__device__ __forceinline__ void sum_cand_slots(const CompressArgs& a, int head, int bx) {
  constexpr int NSF4 = D * D / 4, NF4 = (D * D + 2 * D) / 4;
  const int f4 = bx * 32 + (threadIdx.x >> 3);
  const int sub = threadIdx.x & 7;
  if (f4 >= NF4) return;  // whole groups of eight lanes leave together
  const bool in_S = f4 < NSF4;
  float* base = in_S ? a.spart + (size_t)head * a.nslot * D * D + 4 * f4
                     : a.svkpart + (size_t)head * a.nslot * 2 * D + 4 * (f4 - NSF4);
  const size_t stride = in_S ? (size_t)D * D : (size_t)2 * D;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
  for (int sl = sub; sl < a.nsl1; sl += 8) {
    const float4 p = *reinterpret_cast<const float4*>(base + sl * stride);
    acc.x += p.x; acc.y += p.y; acc.z += p.z; acc.w += p.w;
  }
#pragma unroll
  for (int x = 1; x < 8; x <<= 1) {
    acc.x += __shfl_xor(acc.x, x, 8);
    acc.y += __shfl_xor(acc.y, x, 8);
    acc.z += __shfl_xor(acc.z, x, 8);
    acc.w += __shfl_xor(acc.w, x, 8);
  }
  if (sub == 0) *reinterpret_cast<float4*>(base) = acc;
}

template <int D>
__global__ void __launch_bounds__(256) k_row_combine(CompressArgs a) {
  const int head = blockIdx.y;
  sum_cand_slots<D>(a, head, blockIdx.x);
  if (blockIdx.x == 0) {  // the score producers below add into these
    for (int b = threadIdx.x; b < 2 * TK_HBINS; b += 256)
      a.tk_hh[((size_t)(b / TK_HBINS) * a.H + head) * TK_HBINS + b % TK_HBINS] = 0u;
    if (a.adaptive && head % a.Hkv == 0)
      for (int b = threadIdx.x; b < TK_HBINS; b += 256)
        a.tk_hs[(size_t)(head / a.Hkv) * TK_HBINS + b] = 0u;
  }
  if ((int)blockIdx.x * 32 >= a.R) return;  // uniform over the workgroup
  const int r = blockIdx.x * 32 + (threadIdx.x >> 3);
  const int sub = threadIdx.x & 7;
  float m = -INFINITY, l = 0.f;
  if (r < a.R) {
#pragma unroll 4
    for (int s = sub; s < a.nsl1; s += 8) {
      const float* rp = a.rowpart + (((size_t)head * a.nsl1 + s) * a.R + r) * 2;
      ml_merge(m, l, rp[0], rp[1]);
    }
  }
#pragma unroll
  for (int x = 1; x < 8; x <<= 1) {
    const float m2 = __shfl_xor(m, x), l2 = __shfl_xor(l, x);
    ml_merge(m, l, m2, l2);
  }
  if (r < a.R && sub == 0) {
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
  __shared__ float sAj[kMassMaxTiles * TILE];  // a_j of the slice's tiles
  __shared__ float sRow[512][2];
  __shared__ uint32_t sHist[TK_HBINS];  // keys of the first selection's scores
  __shared__ uint32_t sHistA[TK_HBINS]; // keys of abar (head-adaptive layer-wide selection)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, sl = blockIdx.x;
  const T* Kh = reinterpret_cast<const T*>(a.k) + (size_t)head * a.N * D;
  const int c_lo = a.n_s, c_hi = a.N - a.w;
  const int RT = (a.R + 15) >> 4;
  const float c2 = a.scale * kLog2e;
  const float inv_rows = 1.f / (float)a.R;

  // tiles of this slice that hold candidates (a contiguous range); the next tile's rows
  // are loaded into registers while the current one is consumed.  Every load is issued
  // unconditionally (rows clamped to the last candidate of the slice: rows outside the
  // candidates are never stored) and no global access sits between a prefetch and its
  // use, so the compiler waits for exactly the tile being used; a_j stays in LDS and the
  // pooling, scores and histograms follow the loop.
  const int t_beg = max(sl * a.tps2, c_lo / TILE);
  const int t_end = min(min(sl * a.tps2 + a.tps2, a.ntile), (c_hi + TILE - 1) / TILE);
  const int last_row = max(min(t_end * TILE, c_hi) - 1, 0);
  const int dg = tid % DG;
  typename Frag<T>::type pk[CPT];
  auto load_tile = [&](int t) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int j = min(t * TILE + (tid + 256 * i) / DG, last_row);
      pk[i] = load_frag(Kh + (size_t)j * D + 8 * dg);
    }
  };
  load_tile(t_beg);  // in flight while the row statistics and queries arrive

  for (int r = tid; r < a.R; r += 256) {
    sRow[r][0] = a.rowstat[((size_t)head * a.R + r) * 2 + 0];
    sRow[r][1] = a.rowstat[((size_t)head * a.R + r) * 2 + 1];
  }
  for (int b = tid; b < TK_HBINS; b += 256) sHist[b] = sHistA[b] = 0u;
  // query rows past R repeat row R-1: their terms get weight 0 (and a max of +inf, so
  // that no large logit can overflow into 0 x inf)
  typename Frag<T>::type qf[MTW][KS];
#pragma unroll
  for (int k = 0; k < MTW; ++k) {
    const int mt = wave + 4 * k;
    const T* qrow = window_row<T>(a, head, min(16 * mt + (lane & 15), a.R - 1));
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[k][ks] = load_frag(qrow + 32 * ks + 8 * (lane >> 4));
  }
  __syncthreads();
  float rmax[MTW][4], rinv[MTW][4];  // row statistics of the lane's result rows
#pragma unroll
  for (int k = 0; k < MTW; ++k)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * (wave + 4 * k) + 4 * (lane >> 4) + i;
      const bool ok = r < a.R;
      rmax[k][i] = ok ? sRow[r][0] : INFINITY;
      rinv[k][i] = ok ? sRow[r][1] : 0.f;
    }

  for (int t = t_beg; t < t_end; ++t) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) store_frag(&sK[(tid + 256 * i) / DG][8 * dg], pk[i]);
    load_tile(t + 1);  // past the slice: its last row again
    __syncthreads();
    // each 16-token group's K fragments are read from LDS once for all row tiles
    float col[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      typename Frag<T>::type kb[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kb[ks] = load_frag(&sK[16 * nt + (lane & 15)][32 * ks + 8 * (lane >> 4)]);
#pragma unroll
      for (int k = 0; k < MTW; ++k) {
        if (wave + 4 * k >= RT) continue;
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) mma(acc, qf[k][ks], kb[ks]);
#pragma unroll
        for (int i = 0; i < 4; ++i) col[nt] += fast_exp2(acc[i] * c2 - rmax[k][i]) * rinv[k][i];
      }
    }
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const float x = cross_row_sum(col[nt]);
      if (lane < 16) sA[wave][16 * nt + lane] = x;
    }
    __syncthreads();
    if (tid < TILE)
      sAj[(t - t_beg) * TILE + tid] = (((sA[0][tid] + sA[1][tid]) + sA[2][tid]) + sA[3][tid]) * inv_rows;
  }
  __syncthreads();
  // chunk pooling (chunks are aligned and divide the tile), provisional scores, histograms
  const int tok_beg = t_beg * TILE;
  for (int x = tid; x < (t_end - t_beg) * TILE; x += 256) {
    const int j = tok_beg + x;
    if (j >= c_lo && j < c_hi) {
      const int cs = (j / a.chunk) * a.chunk;
      const int lo = max(cs, c_lo), hi = min(cs + a.chunk, c_hi);
      float s = 0.f;
      for (int i = lo; i < hi; ++i) s += sAj[i - tok_beg];
      const float ab = s / (float)(hi - lo);
      const size_t o = (size_t)head * a.n_c + (j - c_lo);
      const float s0 = ab * a.vnorm[o];
      a.abar[o] = ab;
      a.score0[o] = s0;
      atomicAdd(&sHist[score_key(a.mi_rounds < 0 ? ab : s0) >> 20], 1u);
      if (a.adaptive) atomicAdd(&sHistA[score_key(ab) >> 20], 1u);
    }
  }
  __syncthreads();
  hist_flush<256>(sHist, a.tk_hh + (size_t)head * TK_HBINS);
  if (a.adaptive) hist_flush<256>(sHistA, a.tk_hs + (size_t)(head / a.Hkv) * TK_HBINS);
}

// ------------------------------------------------------------------------------------
// Stage 4/9: per-head selection of the k best scores (ties: lower position first),
// output in ascending position order.  Scores are non-negative floats, so their bit
// patterns (bit 31 clear) order like unsigned integers ("keys").  The kernel producing
// the scores (k_mass, k_residual) also adds each key's bits 30..20 into the head's
// histogram; then two launches over slices of TKS positions spread over all CUs:
//   k_tk_cand   slices x heads: from the head's histogram, the bin B of the k-th largest
//               key and the count of keys above B (every slice finds the same); counts the
//               slice's keys above B and writes its keys inside B (the candidates) in
//               position order;
//   k_tk_write  slices x heads: refines bits 19..10 and 9..0 over the head's candidates
//               (few: one bin spans an eighth of an octave), which gives the k-th key T and
//               how many keys equal to T are kept (the lowest positions); from the per-slice
//               counts it gets its slice's output offset and share of equal keys, then
//               writes the slice's kept positions in order.
// ------------------------------------------------------------------------------------
// Exclusive scan of one int per thread over an NT-thread block; the total goes to *total.
// sW holds 2 * NT / 64 + 1 ints.
template <int NT>
__device__ int block_excl_scan(int x, int* sW, int* total) {
  constexpr int NW = NT / 64;
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
    int v = lane < NW ? sW[lane] : 0;
    int vi = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int y = __shfl_up(vi, o);
      if (lane >= o) vi += y;
    }
    if (lane < NW) sW[NW + lane] = vi - v;  // exclusive wave offsets
    if (lane == NW - 1) sW[2 * NW] = vi;
  }
  __syncthreads();
  const int res = sW[NW + wave] + inc - x;
  *total = sW[2 * NW];
  __syncthreads();
  return res;
}

// Over NB histogram bins in descending order, the bin where the running count reaches
// `need` (1 <= need <= total), found by one wave: lane l holds NB / 64 consecutive bins from
// the top in registers (16-byte LDS reads), one wave scan of their sums, then the lane
// whose range crosses `need` walks its bins.  No block-wide scan or barrier.  Returns
// (bin, count above it) in every lane of the wave.
template <int NB>
__device__ __forceinline__ void wave_find_bin(const uint32_t* hist, int need, uint32_t* bin,
                                              uint32_t* above) {
  constexpr int PER = NB / 64;
  const int lane = threadIdx.x & 63;
  const int lo = NB - PER * (lane + 1);  // the lane's lowest bin
  uint32_t h[PER];
#pragma unroll
  for (int v = 0; v < PER / 4; ++v) {
    const uint4 x = reinterpret_cast<const uint4*>(hist + lo)[v];
    h[4 * v] = x.x; h[4 * v + 1] = x.y; h[4 * v + 2] = x.z; h[4 * v + 3] = x.w;
  }
  int c = 0;
#pragma unroll
  for (int q = 0; q < PER; ++q) c += (int)h[q];
  int inc = c;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o);
    if (lane >= o) inc += y;
  }
  int before = inc - c;
  uint32_t b = 0u, ab = 0u;
  bool found = false;
  const bool mine = before < need && inc >= need;
#pragma unroll
  for (int q = PER - 1; q >= 0; --q) {  // from the lane's top bin down
    if (mine && !found && before + (int)h[q] >= need) {
      b = (uint32_t)(lo + q);
      ab = (uint32_t)before;
      found = true;
    }
    before += (int)h[q];
  }
  const uint64_t m = __ballot(found);
  const int src = m ? (int)__builtin_ctzll(m) : 0;
  *bin = (uint32_t)__shfl((int)b, src);
  *above = (uint32_t)__shfl((int)ab, src);
}

// The TKPT consecutive keys of thread tid in slice sl (positions >= n give valid = false).
// Every read is issued, from a position clamped into the row (the score arrays hold at
// least one entry per row), before the first is used: a read under a per-lane condition
// would be waited for before the next one is issued.
__device__ __forceinline__ void slice_keys(const float* s, int n, int sl, uint32_t (&key)[TKPT],
                                           bool (&valid)[TKPT]) {
  const int j0 = sl * TKS + TKPT * threadIdx.x;
  float v[TKPT];
#pragma unroll
  for (int u = 0; u < TKPT; ++u) v[u] = s[max(min(j0 + u, n - 1), 0)];
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int u = 0; u < TKPT; ++u) {
    valid[u] = j0 + u < n;
    key[u] = valid[u] ? score_key(v[u]) : 0u;
  }
}

__global__ void __launch_bounds__(TKT) k_tk_cand(const float* __restrict__ scores, int n, int k,
                                                   const int* __restrict__ kh,
                                                   const uint32_t* __restrict__ hh,
                                                   int* __restrict__ state,
                                                   int* __restrict__ cnt, uint32_t* __restrict__ cand) {
  __shared__ int sW[2 * (TKT / 64) + 1];
  __shared__ __align__(16) uint32_t hst[TK_HBINS];
  __shared__ uint32_t sh_bin, sh_above;
  const int head = blockIdx.y, sl = blockIdx.x, ntk = gridDim.x;
  if (kh) k = min(kh[head], n);  // head-adaptive count (uniform over the workgroup)
  if (k <= 0) return;
  uint32_t key[TKPT];
  bool valid[TKPT];
  slice_keys(scores + (size_t)head * n, n, sl, key, valid);
  // the head's histogram (every slice workgroup finds the same bin of the k-th key): each
  // thread's bins in 16-byte reads, all issued before the first LDS store
  {
    static_assert(TK_HBINS % (4 * TKT) == 0, "whole 16-byte pieces per thread");
    constexpr int HPT = TK_HBINS / 4 / TKT;
    const uint4* src = reinterpret_cast<const uint4*>(hh + (size_t)head * TK_HBINS);
    uint4 hv[HPT];
#pragma unroll
    for (int u = 0; u < HPT; ++u) hv[u] = src[threadIdx.x + TKT * u];
#pragma unroll
    for (int u = 0; u < HPT; ++u) reinterpret_cast<uint4*>(hst)[threadIdx.x + TKT * u] = hv[u];
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    uint32_t b, ab;
    wave_find_bin<TK_HBINS>(hst, k, &b, &ab);
    if (threadIdx.x == 0) { sh_bin = b; sh_above = ab; }
  }
  __syncthreads();
  const uint32_t B = sh_bin;
  if (sl == 0 && threadIdx.x == 0) {
    state[2 * head] = (int)sh_bin;
    state[2 * head + 1] = (int)sh_above;
  }
  int n_gt = 0, n_c = 0;
#pragma unroll
  for (int u = 0; u < TKPT; ++u) {
    n_gt += valid[u] && (key[u] >> 20) > B;
    n_c += valid[u] && (key[u] >> 20) == B;
  }
  // one scan of both counts, packed in 16-bit halves (a slice holds 2048 positions)
  int tot;
  const int before = block_excl_scan<TKT>(n_gt | (n_c << 16), sW, &tot);
  int pos = before >> 16;
  uint32_t* c = cand + ((size_t)head * ntk + sl) * TKS;
#pragma unroll
  for (int u = 0; u < TKPT; ++u)
    if (valid[u] && (key[u] >> 20) == B) c[pos++] = key[u];
  if (threadIdx.x == 0) {
    cnt[((size_t)head * ntk + sl) * 2] = tot & 0xFFFF;
    cnt[((size_t)head * ntk + sl) * 2 + 1] = tot >> 16;
  }
}

// COV: the same workgroup then adds the covariance and sums of its slice's kept rows
// (negated) or, for a head whose evicted candidates are fewer, of its slice's evicted rows
// into partial slot nsl1 + slice (the work of a separate pass over the selected rows).
template <class T, int D>
__device__ void slice_cov(const CompressArgs& a, int head, int sl, const int32_t* list,
                          int nrows, float sign);

template <class E, int D, bool COV>
__global__ void __launch_bounds__(TKT) k_tk_write(const float* __restrict__ scores, int n, int k,
                                                    const int* __restrict__ kh,
                                                    const int* __restrict__ state,
                                                    const int* __restrict__ cnt,
                                                    const uint32_t* __restrict__ cand,
                                                    int32_t* __restrict__ out, int out_stride,
                                                    int pos_offset, CompressArgs a) {
  __shared__ int s_gt[TK_MAX_SLICES], s_cn[TK_MAX_SLICES], s_gtT[TK_MAX_SLICES], s_eqT[TK_MAX_SLICES];
  __shared__ __align__(16) uint32_t hst[1024];
  __shared__ uint32_t sh_bin, sh_above;
  __shared__ int sW[2 * (TKT / 64) + 1];
  __shared__ int s_off, s_eqb;
  __shared__ int s_start[TK_MAX_SLICES + 1];
  __shared__ uint32_t c_key[TK_CAND_LDS];
  __shared__ uint16_t c_sl[TK_CAND_LDS];
  __shared__ int32_t s_rows[COV ? TKS : 1];  // the slice's rows for the covariance, in order
  __shared__ int s_nrows;
  const int head = blockIdx.y, sl = blockIdx.x, ntk = gridDim.x, tid = threadIdx.x;
  if (kh) k = min(kh[head], n);  // head-adaptive count (uniform over the workgroup)
  if (k <= 0) {
    if constexpr (COV) slice_cov<E, D>(a, head, sl, s_rows, 0, -1.f);  // a zero slot
    return;
  }
  // the slice's own keys are needed last but depend on nothing: requested first
  uint32_t key[TKPT];
  bool valid[TKPT];
  slice_keys(scores + (size_t)head * n, n, sl, key, valid);
  const uint32_t B = (uint32_t)state[2 * head];
  const int above = state[2 * head + 1];
  for (int i = tid; i < ntk; i += TKT) {
    s_gt[i] = cnt[((size_t)head * ntk + i) * 2];
    s_cn[i] = cnt[((size_t)head * ntk + i) * 2 + 1];
    s_gtT[i] = 0;
    s_eqT[i] = 0;
  }
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int i = 0; i < ntk; ++i) { s_start[i] = acc; acc += s_cn[i]; }
    s_start[ntk] = acc;
  }
  __syncthreads();
  // The head's candidates, flattened in slice order, go to LDS with all loads in flight
  // (a flat index finds its slice by bisection over the slice starts); past TK_CAND_LDS
  // candidates the passes read them from global memory instead.
  const int m = s_start[ntk];
  const bool in_lds = m <= TK_CAND_LDS;
  if (in_lds) {
    // the slice of every flat index first (each slice's range filled in LDS), then all
    // loads of the thread, from clamped addresses, then the keys' stores
    for (int s2 = 0; s2 < ntk; ++s2)
      for (int f = s_start[s2] + tid; f < s_start[s2 + 1]; f += TKT) c_sl[f] = (uint16_t)s2;
    __syncthreads();
    constexpr int GU = TK_CAND_LDS / TKT;
    uint32_t v[GU];
#pragma unroll
    for (int u = 0; u < GU; ++u) {
      if (u * TKT < m) {  // uniform
        const int f = min(u * TKT + tid, m - 1);
        const int s2 = c_sl[f];
        v[u] = cand[((size_t)head * ntk + s2) * TKS + (f - s_start[s2])];
      }
    }
#pragma unroll
    for (int u = 0; u < GU; ++u) {
      const int f = u * TKT + tid;
      if (f < m) c_key[f] = v[u];
    }
  }
  __syncthreads();
  auto for_each_cand = [&](auto&& fn) {
    if (in_lds) {
      for (int f = tid; f < m; f += TKT) fn(c_key[f], (int)c_sl[f]);
    } else {
      for (int s2 = 0; s2 < ntk; ++s2) {
        const uint32_t* c = cand + ((size_t)head * ntk + s2) * TKS;
        for (int i = tid; i < s_cn[s2]; i += TKT) fn(c[i], s2);
      }
    }
  };
  // bits 19..10, then 9..0, over the candidates (all of them have bits 30..20 = B)
  uint32_t prefix = B << 20, mask = 0x7FF00000u;
  int remaining = k - above;
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 10 : 0;
    for (int i = tid; i < 1024; i += TKT) hst[i] = 0;
    __syncthreads();
    for_each_cand([&](uint32_t key, int) {
      if ((key & mask) == prefix) atomicAdd(&hst[(key >> shift) & 1023u], 1u);
    });
    __syncthreads();
    if (tid < 64) {
      uint32_t b, ab;
      wave_find_bin<1024>(hst, remaining, &b, &ab);
      if (tid == 0) { sh_bin = b; sh_above = ab; }
    }
    __syncthreads();
    prefix |= sh_bin << shift;
    mask |= 1023u << shift;
    remaining -= (int)sh_above;
    __syncthreads();  // hst is cleared again by the next pass
  }
  const uint32_t T = prefix;
  const int need = remaining;  // keys equal to T to keep (>= 1), the lowest positions
  // per slice: candidates above T and equal to T
  for_each_cand([&](uint32_t key, int s2) {
    if (key > T) atomicAdd(&s_gtT[s2], 1);
    else if (key == T) atomicAdd(&s_eqT[s2], 1);
  });
  __syncthreads();
  const bool direct = n - k < k;  // the head's evicted candidates are the fewer
  if (tid == 0) {  // fixed order over the slices
    int eb = 0, ob = 0;
    for (int s2 = 0; s2 < ntk; ++s2) {
      const int kept_s2 = s_gt[s2] + s_gtT[s2] + min(max(need - eb, 0), s_eqT[s2]);
      if (s2 == sl) {
        s_off = ob;
        s_eqb = eb;
        const int valid_s2 = min(TKS, n - s2 * TKS);
        s_nrows = direct ? valid_s2 - kept_s2 : kept_s2;
      }
      ob += kept_s2;
      eb += s_eqT[s2];
    }
  }
  __syncthreads();
  // the slice's kept positions, in order: one scan of (keys above T, keys at T) per
  // thread, packed in 16-bit halves; the keys at T kept before a thread are the first of
  // the need - (keys at T in earlier slices) still to keep
  int n_gt = 0, n_eq = 0;
#pragma unroll
  for (int u = 0; u < TKPT; ++u) {
    n_gt += valid[u] && key[u] > T;
    n_eq += valid[u] && key[u] == T;
  }
  int tot;
  const int before = block_excl_scan<TKT>(n_gt | (n_eq << 16), sW, &tot);
  int eq_rank = s_eqb + (before >> 16);
  bool keep[TKPT];
#pragma unroll
  for (int u = 0; u < TKPT; ++u) {
    const bool eq = valid[u] && key[u] == T;
    keep[u] = (valid[u] && key[u] > T) || (eq && eq_rank < need);
    eq_rank += eq;
  }
  // p = kept positions before the thread's current one, so a position that is not kept
  // is the (j - p)-th evicted one
  int p = s_off + (before & 0xFFFF) + min(max(need - s_eqb, 0), before >> 16);
  int32_t* o = out + (size_t)head * out_stride;
  const int j0 = sl * TKS + TKPT * tid;
  const int e_off = sl * TKS - s_off;  // evicted positions before the slice
#pragma unroll
  for (int u = 0; u < TKPT; ++u) {
    if (keep[u]) {
      if (p < k) {
        o[p] = j0 + u + pos_offset;
        if (COV && !direct) s_rows[min(max(p - s_off, 0), TKS - 1)] = j0 + u + pos_offset;
      }
      ++p;
    } else if (COV && valid[u] && direct) {  // not kept: the (j - p)-th evicted position
      const int e = j0 + u - p;
      if (e >= 0 && e < n - k) s_rows[min(max(e - e_off, 0), TKS - 1)] = j0 + u + pos_offset;
    }
  }
  if constexpr (COV) {
    __syncthreads();
    slice_cov<E, D>(a, head, sl, s_rows, min(s_nrows, TKS), direct ? 1.f : -1.f);
  }
}

// ------------------------------------------------------------------------------------
// Stage 6/11: covariance and sums of one head's kept rows (stored negated) or, when they
// are fewer, of its evicted rows (stored as they are), read through their positions, into
// the slots after the candidate slices.
// ------------------------------------------------------------------------------------
// Rows list[row0 + 2p] and list[row0 + 2p + 1] of K and V (head base pointers), list
// entries clamped to the n_rows given and the positions to the head's N rows; issued as
// tile_load issues its rows.
template <class T, int D, int NT>
__device__ __forceinline__ void tile_load_list(TileRegs<T, D, NT>& R, const T* Kh, const T* Vh,
                                               const int32_t* list, int row0, int n_rows, int N,
                                               int tid) {
  typedef TileRegs<T, D, NT> TR;
  const int col = 8 * TR::group(tid);
#pragma unroll
  for (int i = 0; i < TR::NP; ++i) {
    const int p = TR::pair(tid, i);
    const int j0 = min(max(list[min(row0 + 2 * p, n_rows - 1)], 0), N - 1);
    const int j1 = min(max(list[min(row0 + 2 * p + 1, n_rows - 1)], 0), N - 1);
    R.k[i][0] = load_frag(Kh + (size_t)j0 * D + col);
    R.k[i][1] = load_frag(Kh + (size_t)j1 * D + col);
    R.v[i][0] = load_frag(Vh + (size_t)j0 * D + col);
    R.v[i][1] = load_frag(Vh + (size_t)j1 * D + col);
  }
}

// Covariance and sums of `nrows` rows of head `head` (positions list[0..nrows), LDS or
// global), written with `sign` into partial slot nsl1 + sl; 256 threads.
template <class T, int D>
__device__ void slice_cov(const CompressArgs& a, int head, int sl, const int32_t* list,
                          int nrows, float sign) {
  constexpr int NT = 256, NW = 4;
  constexpr bool BF = sizeof(T) == 2;  // bf16: K and V tiles as they are (transposed reads)
  constexpr int PAD = 16 / (int)sizeof(T);
  constexpr int LDT = TILE + PAD, LDN = D + 16;
  constexpr int QM = CovSplit<D, NW>::QM, QN = CovSplit<D, NW>::QN;
  typedef TileRegs<T, D, NT> TR;
  __shared__ __align__(16) T sKT[BF ? TILE : D][BF ? LDN : LDT];  // bf16: K rows; fp32: K^T
  __shared__ __align__(16) T sVT[BF ? TILE : D][BF ? LDN : LDT];  // bf16: V rows; fp32: V^T
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const T* Kh = reinterpret_cast<const T*>(a.k) + (size_t)head * a.N * D;
  const T* Vh = reinterpret_cast<const T*>(a.v) + (size_t)head * a.N * D;
  f32x4 cacc[QM][QN];
#pragma unroll
  for (int mi = 0; mi < QM; ++mi)
#pragma unroll
    for (int ni = 0; ni < QN; ++ni) cacc[mi][ni] = zero4();
  float sk[8], sv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) sk[e] = sv[e] = 0.f;
  auto in_rows = [&](int j) { return j < nrows; };
  const int ntiles = (nrows + TILE - 1) / TILE;
  TR R;
  if (ntiles > 0) tile_load_list<T, D, NT>(R, Kh, Vh, list, 0, nrows, a.N, tid);
  for (int t = 0; t < ntiles; ++t) {
    float ss[TR::NP][2];
    R.arrive();
    if constexpr (BF) {
      if (TR::active(tid)) {
#pragma unroll
        for (int i = 0; i < TR::NP; ++i) {
          const int p = TR::pair(tid, i);
          store_frag(&sKT[2 * p][8 * TR::group(tid)], R.k[i][0]);
          store_frag(&sKT[2 * p + 1][8 * TR::group(tid)], R.k[i][1]);
        }
      }
      tile_sums_nat<D, NT, LDN>(R, sVT, t * TILE, in_rows, sk, sv, ss, tid);
    } else {
      tile_store_t<T, D, NT, LDT>(R, sKT, sVT, t * TILE, in_rows, sk, sv, ss, tid);
    }
    if (t + 1 < ntiles) tile_load_list<T, D, NT>(R, Kh, Vh, list, (t + 1) * TILE, nrows, a.N, tid);
    __syncthreads();
    if constexpr (BF)
      cov_tile_tr<D, NW>(&sVT[0][0], &sKT[0][0], LDN, cacc, wave, lane);
    else
      cov_tile<T, D, NW, LDT>(sVT, sKT, cacc, wave, lane);
    __syncthreads();
  }
  write_cov_partials<T, D, NT>(a, head, a.nsl1 + sl, cacc, sv, sk, sign,
                              reinterpret_cast<float*>(&sVT[0][0]), tid);
}

// ------------------------------------------------------------------------------------
// Stage 7/12: fixed-order sum of the partial slots -> raw S, s_v, s_k of the evicted set
// (stage 7: the provisional set, into the workspace; stage 12: the output moments): the
// candidates' sums (slot 0, where the row-statistics launch has added up the candidate
// slots) and the selection's slots, or only the evicted rows' slots of a head that sums
// them directly.  Eight lanes per float4 of a head's D*D + 2D values, lane `sub` summing
// the listed slots sub, sub + 8, ..., then a fixed xor tree across the eight lanes.
// ------------------------------------------------------------------------------------
// S_bf16: S_out holds bf16 (each fp32 sum rounded once, to nearest even).
template <int D>
__device__ __forceinline__ void reduce_slots(const CompressArgs& a, int head, int bx, void* S_out,
                                             bool S_bf16, float* sv_out, float* sk_out,
                                             int32_t* ne_out) {
  constexpr int NSF4 = D * D / 4, NF4 = (D * D + 2 * D) / 4;
  const int f4 = bx * 32 + (threadIdx.x >> 3);
  const int sub = threadIdx.x & 7;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  // listed slots: u = 0 is slot 0 (the candidates' sums) unless the head sums directly,
  // then the selection's slots nsl1 ... nslot - 1
  const int lead = direct_sums(a, head) ? 0 : 1;
  const int n_use = a.nslot - a.nsl1 + lead;
  if (f4 < NF4) {
    const bool in_S = f4 < NSF4;
    const float* base = in_S ? a.spart + (size_t)head * a.nslot * D * D + 4 * f4
                             : a.svkpart + (size_t)head * a.nslot * 2 * D + 4 * (f4 - NSF4);
    const size_t stride = in_S ? (size_t)D * D : (size_t)2 * D;
#pragma unroll 4
    for (int u = sub; u < n_use; u += 8) {
      const int sl = u < lead ? 0 : a.nsl1 + u - lead;
      const float4 p = *reinterpret_cast<const float4*>(base + sl * stride);
      acc.x += p.x; acc.y += p.y; acc.z += p.z; acc.w += p.w;
    }
  }
#pragma unroll
  for (int x = 1; x < 8; x <<= 1) {
    acc.x += __shfl_xor(acc.x, x);
    acc.y += __shfl_xor(acc.y, x);
    acc.z += __shfl_xor(acc.z, x);
    acc.w += __shfl_xor(acc.w, x);
  }
  if (f4 < NF4 && sub == 0) {
    if (f4 < NSF4 && S_bf16) {
      bf16_t* dst = static_cast<bf16_t*>(S_out) + (size_t)head * D * D + 4 * f4;
      *reinterpret_cast<uint2*>(dst) = make_uint2(bf16_pair(acc.x, acc.y), bf16_pair(acc.z, acc.w));
    } else {
      float* dst;
      if (f4 < NSF4) {
        dst = static_cast<float*>(S_out) + (size_t)head * D * D + 4 * f4;
      } else {
        const int e = 4 * (f4 - NSF4);  // [0, D): s_v, [D, 2D): s_k
        dst = e < D ? sv_out + (size_t)head * D + e : sk_out + (size_t)head * D + (e - D);
      }
      *reinterpret_cast<float4*>(dst) = acc;
    }
  }
  if (ne_out && bx == 0 && threadIdx.x == 0) ne_out[head] = a.n_c - head_keep(a, head);
}

// Also clears the head's histogram of the moment round that follows (the round before
// filled it, and its selection has read it).
template <int D>
__global__ void __launch_bounds__(256) k_reduce(CompressArgs a, float* S_out, float* sv_out,
                                                 float* sk_out, int32_t* ne_out) {
  reduce_slots<D>(a, blockIdx.y, blockIdx.x, S_out, false, sv_out, sk_out, ne_out);
  if (blockIdx.x == 0)
    for (int b = threadIdx.x; b < TK_HBINS; b += 256)
      a.tk_hh[((size_t)a.H + blockIdx.y) * TK_HBINS + b] = 0u;
}

// ------------------------------------------------------------------------------------
// Stage 8: moment residual score of every candidate (Sec. 4.2 Eq. residual).
// Wave w owns rows [32w, 32w+32) of S_tilde0 (D = 128; 16 rows for D = 64), built in
// registers from the raw provisional sums (centring and clamp, App. A.1 Eq. app_S_tilde,
// App. C.2) and kept as MFMA A fragments: fp32, or a bf16 hi/lo pair whose two products
// add up to fp32-level accuracy.  Candidate tiles of 64 rows of K and V stream through
// LDS (natural layout) with the next tile prefetched into registers.  Each wave forms
// S_tilde0 k_j for its rows, the partial ||v_j - v_bar - c S_tilde0 k_j||^2 over them, and
// the four partials are added in wave order.
// ------------------------------------------------------------------------------------
template <class T, int D>
__global__ void __launch_bounds__(256, sizeof(T) == 2 ? 2 : 1) k_residual(CompressArgs a) {
  constexpr int KS = D / 32, DG = D / 8, PAD = 16 / (int)sizeof(T);
  constexpr int LDK = D + PAD;
  constexpr int CPT = TILE * DG / 256;
  constexpr bool BF = sizeof(T) == 2;
  constexpr int NPL = BF ? 2 : 1;          // A fragment planes: bf16 hi + lo, or fp32
  constexpr int MTPW = D / 64;             // 16-row tiles of S_tilde0 per wave
  typedef typename Frag<T>::type FragT;
  __shared__ __align__(16) T sK[TILE][LDK];
  __shared__ __align__(16) T sV[TILE][LDK];
  __shared__ float sRho[4][TILE];
  __shared__ float sRes[kResMaxTiles * TILE];  // squared residual norms of the slice
  __shared__ float sSv[D], sSk[D];
  __shared__ uint32_t sHist[TK_HBINS];  // keys of the final selection's scores
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int b = tid; b < TK_HBINS; b += 256) sHist[b] = 0u;
  const int head = blockIdx.y, sl = blockIdx.x;
  const int c_lo = a.n_s, c_hi = a.N - a.w;
  const float n0 = (float)(a.n_c - head_keep(a, head));  // 0: everything kept, empty summary
  const float inv_n = n0 > 0.f ? 1.f / n0 : 0.f;
  const float coef = n0 > 0.f ? a.scale / n0 : 0.f;
  const T* Kh = reinterpret_cast<const T*>(a.k) + (size_t)head * a.N * D;
  const T* Vh = reinterpret_cast<const T*>(a.v) + (size_t)head * a.N * D;

  // Candidate tiles of this slice; the next tile's rows are loaded into registers while
  // the current one is consumed.  Every load is issued unconditionally (rows clamped to
  // the slice's last candidate: rows past it are never stored) and no global access sits
  // between a prefetch and its use, so the compiler waits for exactly the tile being
  // used; the norms stay in LDS and the scores and histogram follow the loop.
  const int n_tiles = (a.n_c + TILE - 1) / TILE;
  const int t_beg = sl * a.tps3, t_end = min(t_beg + a.tps3, n_tiles);
  const int last_row = max(min(c_lo + t_end * TILE, c_hi) - 1, 0);
  const int dg = tid % DG;
  FragT pk[CPT], pv[CPT];
  auto load_tile = [&](int t) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int j = min(c_lo + t * TILE + (tid + 256 * i) / DG, last_row);
      pk[i] = load_frag(Kh + (size_t)j * D + 8 * dg);
      pv[i] = load_frag(Vh + (size_t)j * D + 8 * dg);
    }
  };
  load_tile(t_beg);  // in flight while the summary is formed

  for (int t = tid; t < D; t += 256) {
    sSv[t] = a.sv0[(size_t)head * D + t];
    sSk[t] = a.sk0[(size_t)head * D + t];
  }
  __syncthreads();
  // A fragments: row 16*(MTPW*wave + m) + lane%16, columns 32*ks + 8*(lane/16) + e
  FragT af[MTPW][KS][NPL];
  const float* S0 = a.s0 + (size_t)head * D * D;
  f32x8 raw[MTPW][KS];  // every read issued before the first is used (one round trip)
#pragma unroll
  for (int m = 0; m < MTPW; ++m)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      raw[m][ks] = load_frag(S0 + (size_t)(16 * (MTPW * wave + m) + (lane & 15)) * D + 32 * ks +
                             8 * (lane >> 4));
#pragma unroll
  for (int m = 0; m < MTPW; ++m) {
    const int row = 16 * (MTPW * wave + m) + (lane & 15);
    const float sv = sSv[row];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int col = 32 * ks + 8 * (lane >> 4);
      float st[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        st[e] = raw[m][ks][e] - sv * sSk[col + e] * inv_n;
        if (fabsf(st[e]) < a.tau) st[e] = 0.f;
      }
      if constexpr (BF) {
        u32x4 hi, lo;
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          uint32_t h, l;
          bf16_split_pair(st[e], st[e + 1], h, l);
          hi[e / 2] = h;
          lo[e / 2] = l;
        }
        af[m][ks][0] = __builtin_bit_cast(FragT, hi);
        af[m][ks][NPL - 1] = __builtin_bit_cast(FragT, lo);
      } else {
        f32x8 f;
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = st[e];
        af[m][ks][0] = __builtin_bit_cast(FragT, f);
      }
    }
  }
  // r = v - coef (v_bar0 / coef + S_tilde0 k): the accumulators start at v_bar0 / coef =
  // s_v0 / scale for this lane's result rows 16*(MTPW*wave + m) + 4*(lane/16) + i, so the
  // mean comes out of the MFMAs
  float vb[MTPW][4];
#pragma unroll
  for (int m = 0; m < MTPW; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      vb[m][i] = n0 > 0.f ? sSv[16 * (MTPW * wave + m) + 4 * (lane >> 4) + i] / a.scale : 0.f;

  for (int t = t_beg; t < t_end; ++t) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int tt = (tid + 256 * i) / DG;
      store_frag(&sK[tt][8 * dg], pk[i]);
      store_frag(&sV[tt][8 * dg], pv[i]);
    }
    load_tile(t + 1);  // past the slice: its last row again
    __syncthreads();
    FragT bfr[4][KS];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        bfr[nt][ks] = load_frag(&sK[16 * nt + (lane & 15)][32 * ks + 8 * (lane >> 4)]);
    float rho[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < MTPW; ++m) {
      f32x4 acc[4];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[nt][i] = vb[m][i];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int pl = 0; pl < NPL; ++pl)
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) mma(acc[nt], af[m][ks][pl], bfr[nt][ks]);
      const int a0 = 16 * (MTPW * wave + m) + 4 * (lane >> 4);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        float v[4];
        load4(&sV[16 * nt + (lane & 15)][a0], v);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float r = fmaf(-coef, acc[nt][i], v[i]);
          rho[nt] = fmaf(r, r, rho[nt]);
        }
      }
    }
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const float x = cross_row_sum(rho[nt]);
      if (lane < 16) sRho[wave][16 * nt + lane] = x;
    }
    __syncthreads();
    if (tid < TILE)
      sRes[(t - t_beg) * TILE + tid] = ((sRho[0][tid] + sRho[1][tid]) + sRho[2][tid]) + sRho[3][tid];
  }
  __syncthreads();
  for (int x = tid; x < (t_end - t_beg) * TILE; x += 256) {
    const int j = c_lo + t_beg * TILE + x;
    if (j < c_hi) {
      const size_t o = (size_t)head * a.n_c + (j - c_lo);
      const float sc = a.abar[o] * sqrtf(sRes[x]);
      a.score[o] = sc;
      atomicAdd(&sHist[score_key(sc) >> 20], 1u);
    }
  }
  __syncthreads();
  hist_flush<256>(sHist, a.tk_hh + ((size_t)a.H + head) * TK_HBINS);
}

// ------------------------------------------------------------------------------------
// Stage 10: retained rows (sinks, kept candidates, window) -> k_out/v_out, idx, lens.
// With budget >= N every row is retained.
// ------------------------------------------------------------------------------------
template <class T, int D>
__device__ __forceinline__ void gather_out(const CompressArgs& a, int head, int bx, int n_out,
                                           int keep_all) {
  constexpr int DG = D / 8;
  const int c = bx * 256 + threadIdx.x;
  const int i = c / DG, dg = c % DG;
  const int kk = keep_all ? 0 : head_keep(a, head);
  if (!keep_all && a.kh) n_out = a.n_s + kk + a.w;  // head-adaptive: this head's length
  if (bx == 0 && threadIdx.x == 0) a.lens_out[head] = n_out;
  if (i >= n_out) return;
  int pos;
  if (keep_all || i < a.n_s) pos = i;
  else if (i < a.n_s + kk) pos = a.kept[(size_t)head * a.kmax + (i - a.n_s)];
  else pos = a.N - a.w + (i - a.n_s - kk);
  pos = min(max(pos, 0), a.N - 1);  // a kept position is an address: never outside the rows
  const size_t src = ((size_t)head * a.N + pos) * D + 8 * dg;
  const size_t dst = ((size_t)head * a.cap + i) * D + 8 * dg;
  store_frag(reinterpret_cast<T*>(a.k_out) + dst, load_frag(reinterpret_cast<const T*>(a.k) + src));
  store_frag(reinterpret_cast<T*>(a.v_out) + dst, load_frag(reinterpret_cast<const T*>(a.v) + src));
  if (dg == 0) a.idx_out[(size_t)head * a.idx_stride + i] = pos;
}

template <class T, int D>
__global__ void __launch_bounds__(256) k_gather_out(CompressArgs a, int n_out, int keep_all) {
  gather_out<T, D>(a, blockIdx.y, blockIdx.x, n_out, keep_all);
}

// The last launch: the first reduce_blocks<D>() workgroups of each head sum the final
// selection's slots into the output moments, the others copy the retained rows.
template <class T, int D>
__global__ void __launch_bounds__(256) k_finish(CompressArgs a, int n_out) {
  const int head = blockIdx.y;
  constexpr int RB = reduce_blocks<D>();
  if ((int)blockIdx.x < RB) reduce_slots<D>(a, head, blockIdx.x, a.S, a.S_bf16, a.s_v, a.s_k, a.n_e);
  else gather_out<T, D>(a, head, blockIdx.x - RB, n_out, 0);
}

template <int D>
__global__ void __launch_bounds__(256) k_zero_moments(CompressArgs a) {
  const int head = blockIdx.y;
  for (int e = blockIdx.x * 256 + threadIdx.x; e < D * D; e += gridDim.x * 256) {
    if (a.S_bf16) static_cast<bf16_t*>(a.S)[(size_t)head * D * D + e] = 0;
    else static_cast<float*>(a.S)[(size_t)head * D * D + e] = 0.f;
  }
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

// `which` selects the histogram the score producer filled (0: first selection, 1: final).
// The selection's covariance slots are written by the same launch (k_tk_write<.., true>).
template <class T, int D>
static hipError_t launch_topk(const CompressArgs& a, const float* scores, int which,
                              int32_t* out, hipStream_t st) {
  if (a.k_keep <= 0) return hipSuccess;
  const dim3 grid(a.ntk, a.H);
  hipLaunchKernelGGL(k_tk_cand, grid, dim3(TKT), 0, st, scores, a.n_c, a.k_keep,
                     (const int*)a.kh, (const uint32_t*)(a.tk_hh + (size_t)which * a.H * TK_HBINS),
                     a.tk_state, a.tk_cnt, a.tk_cand);
  MKV_CHECK_LAUNCH();
  hipLaunchKernelGGL((k_tk_write<T, D, true>), grid, dim3(TKT), 0, st, scores, a.n_c, a.k_keep,
                     (const int*)a.kh, (const int*)a.tk_state, (const int*)a.tk_cnt,
                     (const uint32_t*)a.tk_cand, out, a.kmax, a.n_s, a);
  MKV_CHECK_LAUNCH();
  return hipSuccess;
}

// Head-adaptive budgets: one layer-wide selection per sequence over the Hkv heads' abar
// rows (contiguous in memory, position head * n_c + j), the Hkv * k_keep largest with
// equal values in (head, position) order; then each head's share of them.
__global__ void __launch_bounds__(64) k_ada_counts(CompressArgs a) {
  const int b = blockIdx.x;
  const int K = a.Hkv * a.k_keep;
  const int32_t* o = a.kept_all + (size_t)b * K;
  auto lower = [&](int x) {  // first index with o[i] >= x (o ascending)
    int lo = 0, hi = K;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (o[mid] < x) lo = mid + 1; else hi = mid;
    }
    return lo;
  };
  for (int h = threadIdx.x; h < a.Hkv; h += 64)
    a.kh[(size_t)b * a.Hkv + h] = lower((h + 1) * a.n_c) - lower(h * a.n_c);
}

static hipError_t launch_head_budgets(const CompressArgs& a, hipStream_t st) {
  if (!a.adaptive || a.k_keep <= 0) return hipSuccess;
  const int n = a.Hkv * a.n_c, k = a.Hkv * a.k_keep;
  const dim3 grid(a.ntk_g, a.B);
  hipLaunchKernelGGL(k_tk_cand, grid, dim3(TKT), 0, st, (const float*)a.abar, n, k,
                     (const int*)nullptr, (const uint32_t*)a.tk_hs, a.tk_state_g, a.tk_cnt_g,
                     a.tk_cand_g);
  MKV_CHECK_LAUNCH();
  hipLaunchKernelGGL((k_tk_write<float, 64, false>), grid, dim3(TKT), 0, st, (const float*)a.abar, n, k,
                     (const int*)nullptr, (const int*)a.tk_state_g, (const int*)a.tk_cnt_g,
                     (const uint32_t*)a.tk_cand_g, a.kept_all, k, 0, a);
  MKV_CHECK_LAUNCH();
  hipLaunchKernelGGL(k_ada_counts, dim3(a.B), dim3(64), 0, st, a);
  MKV_CHECK_LAUNCH();
  return hipSuccess;
}

template <class T, int D, int MTW>
static hipError_t run_compress(const CompressArgs& a, hipStream_t st, float* dbg_abar,
                               float* dbg_score0, float* dbg_score, int32_t* dbg_kept0) {
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
  hipLaunchKernelGGL((k_rows_cov<T, D, MTW>), dim3(a.nsl1, H), dim3(RC_THREADS), 0, st, a);
  MKV_CHECK_LAUNCH();
  hipLaunchKernelGGL((k_row_combine<D>), dim3(std::max((a.R + 31) / 32, reduce_blocks<D>()), H), blk, 0, st, a);
  MKV_CHECK_LAUNCH();
  hipLaunchKernelGGL((k_mass<T, D, 2 * MTW>), dim3(a.nsl2, H), blk, 0, st, a);
  MKV_CHECK_LAUNCH();
  hipError_t te = launch_head_budgets(a, st);
  if (te != hipSuccess) return te;
  const float* first_scores = a.mi_rounds < 0 ? a.abar : a.score0;
  int32_t* first_out = a.mi_rounds >= 1 ? a.kept0 : a.kept;
  te = launch_topk<T, D>(a, first_scores, 0, first_out, st);
  if (te != hipSuccess) return te;
  // moment rounds: the previous selection's slots give its evicted set's moments, which
  // score the candidates again; every round's selection rewrites the slots
  for (int r = 1; r <= a.mi_rounds; ++r) {
    hipLaunchKernelGGL((k_reduce<D>), dim3(reduce_blocks<D>(), H), blk, 0, st, a, a.s0, a.sv0,
                       a.sk0, (int32_t*)nullptr);
    MKV_CHECK_LAUNCH();
    hipLaunchKernelGGL((k_residual<T, D>), dim3(a.nsl3, H), blk, 0, st, a);
    MKV_CHECK_LAUNCH();
    te = launch_topk<T, D>(a, a.score, 1, a.kept, st);
    if (te != hipSuccess) return te;
  }
  const int n_out_max = a.kh ? a.n_s + a.w + a.kmax : a.L;  // the longest head's rows
  hipLaunchKernelGGL((k_finish<T, D>), dim3(reduce_blocks<D>() + (n_out_max * (D / 8) + 255) / 256, H),
                     blk, 0, st, a, a.L);
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
    const size_t rows = a.kh ? a.kmax : a.k_keep;
    if (hipMemcpy2DAsync(dbg_kept0, rows * 4, src, (size_t)a.kmax * 4, rows * 4,
                         H, hipMemcpyDeviceToDevice, st) != hipSuccess)
      return hipGetLastError();
  }
  return hipSuccess;
}

template <class T, int D>
static hipError_t run_compress_r(const CompressArgs& a, hipStream_t st, float* d0, float* d1,
                                 float* d2, int32_t* d3) {
  const int rt = (a.R + 15) / 16;         // 16-row tiles of window queries
  if (rt <= 8) return run_compress<T, D, 1>(a, st, d0, d1, d2, d3);
  if (rt <= 16) return run_compress<T, D, 2>(a, st, d0, d1, d2, d3);
  return run_compress<T, D, 4>(a, st, d0, d1, d2, d3);
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
