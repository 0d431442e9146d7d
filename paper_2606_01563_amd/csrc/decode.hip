// Corrected decode attention over the retained cache (Algorithm 1 Phase 2; Eqs. fhat,
// jensen and fused; log-domain mixing weight of App. C.2), split-K over the cache.
//
// k_decode<.., FUSED = false>  grid (nsplit, B*Hkv), 256 threads.  Each workgroup streams
//                 one slice of one KV head's retained rows for all G query heads of the
//                 group: Q.K^T on MFMA (the G queries padded to 16 rows), online softmax in
//                 the base-2 domain, P.V on the vector ALU over coalesced rows, the next
//                 16-row block prefetched while the current one is consumed.  It also
//                 computes its share of the rows of S_tilde q (clamped covariance times
//                 each query) on fp32 MFMA, so the d x d summary is read once per head in
//                 total.  The new token (if any) is appended by the workgroup owning its row.
// k_decode_merge  one wave per (b, query head): merges the slices in a fixed order
//                 (f_R, log Z_R), mixes in the first-order estimate f_E_hat with the Jensen
//                 weight, writes the outputs and bumps lens after an append.
// k_decode<.., FUSED = true>   one workgroup per KV head (nsplit = 1): the same stream,
//                 then the merge and the correction in the epilogue, no second launch.
// A same-launch "last workgroup merges" scheme for nsplit > 1 would need a device-scope
// release/acquire in every workgroup, which on this multi-XCD part is a whole-L2
// write-back and invalidate per wave; the merge is therefore a separate launch.
#include "mkv_device.h"
#include "mkv_launch.h"

namespace mkv {

// Rows [r0, r1) of S_tilde q for the G queries of one KV head (unscaled), on fp32 MFMA:
// A = 16-row tiles of S_tilde = S - s_v s_k^T / n_e, centred and clamped as they are
// loaded; B = the queries as fp32 (query g in column g).  Wave w takes the tiles starting
// at r0 + 16w, r0 + 16w + 64, ...; result (g, r) goes to dst[g * D + r].
template <class T, int D>
__device__ __forceinline__ void stilde_q(const DecodeArgs& a, int head, const T* qh, int G,
                                         int r0, int r1, int wave, int lane, float inv_n,
                                         float* dst) {
  constexpr int KS = D / 32;
  const float* Sh = a.S + (size_t)head * D * D;
  const float* skh = a.s_k + (size_t)head * D;
  const float* svh = a.s_v + (size_t)head * D;
  const int g = lane & 15;
  f32x8 qb[KS];
  float skc[KS][8];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int col = 32 * ks + 8 * (lane >> 4) + e;
      qb[ks][e] = g < G ? to_f(qh[(size_t)g * D + col]) : 0.f;
      skc[ks][e] = skh[col] * inv_n;
    }
  for (int m0 = r0 + 16 * wave; m0 < r1; m0 += 64) {
    const int row = m0 + (lane & 15);
    const bool ok = row < r1;
    const float sv = ok ? svh[row] : 0.f;
    f32x8 raw[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      raw[ks] = ok ? load_frag(Sh + (size_t)row * D + 32 * ks + 8 * (lane >> 4)) : zero_frag<float>();
    f32x4 acc = zero4();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      f32x8 af;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float st = raw[ks][e] - sv * skc[ks][e];
        af[e] = fabsf(st) < a.tau ? 0.f : st;
      }
      mma(acc, af, qb[ks]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = m0 + 4 * (lane >> 4) + i;
      if (g < G && r < r1) dst[(size_t)g * D + r] = acc[i];
    }
  }
}

// log Z_R from the merged (max in log2 units, sum) and the Jensen mixing weight w_R.
struct Mix {
  float log_zr, w_r;
};
__device__ __forceinline__ Mix mix_weights(float M, float l, int ne, float q_dot_sk,
                                           float scale) {
  Mix r;
  r.log_zr = (l > 0.f) ? (M + __log2f(l)) * kLn2 : -INFINITY;
  r.w_r = 1.f;
  if (ne > 0) {
    const float log_ze = logf((float)ne) + scale * q_dot_sk / (float)ne;  // Jensen estimate
    const float hi = fmaxf(r.log_zr, log_ze);
    const float lse = hi + logf(expf(r.log_zr - hi) + expf(log_ze - hi));
    r.w_r = expf(r.log_zr - lse);
  }
  return r;
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Two tokens' values of one V column packed for the transposed LDS tile.
__device__ __forceinline__ void store_vpair(bf16_t* p, uint32_t lo_dw, uint32_t hi_dw, int h) {
  *reinterpret_cast<uint32_t*>(p) = __builtin_amdgcn_perm(hi_dw, lo_dw, h ? 0x07060302u : 0x05040100u);
}

template <class T, int D, int GMAX, bool FUSED>
__global__ void __launch_bounds__(256) k_decode(DecodeArgs a) {
  constexpr int KS = D / 32;        // MFMA contraction steps per row
  constexpr int TB = 32;            // tokens per wave iteration
  constexpr int DG = D / 8;         // 8-column groups of a row
  constexpr int NVC = DG / 4;       // V chunks (16 or 32 bytes) per lane and token
  constexpr int NT = D / 16;        // 16-column output tiles of P.V
  constexpr int PT = 16 / (int)sizeof(T);  // row padding (16 bytes)
  static_assert(GMAX <= 16, "G <= 16");
  typedef typename Frag<T>::type FragT;

  __shared__ __align__(16) T s_vt[4][D][TB + PT];     // per-wave V^T tile
  __shared__ __align__(16) T s_p[4][16][TB + PT];     // per-wave P (A operand of P.V)
  __shared__ float s_o[4][GMAX][D];
  __shared__ float s_m[4][GMAX];
  __shared__ float s_l[4][GMAX];
  __shared__ float s_sq[FUSED ? GMAX : 1][FUSED ? D : 1];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int head = blockIdx.y;          // b * Hkv + h
  const int split = blockIdx.x;
  const int G = a.G;
  const int b = head / a.Hkv, h = head % a.Hkv;
  const size_t cache_off = (size_t)head * a.cap * D;
  T* const k_cache = reinterpret_cast<T*>(a.k_cache);
  T* const v_cache = reinterpret_cast<T*>(a.v_cache);
  const T* kc = k_cache + cache_off;
  const T* vc = v_cache + cache_off;
  const T* qh = reinterpret_cast<const T*>(a.q) + ((size_t)b * a.Hkv * G + (size_t)h * G) * D;

  const int old_len = a.lens[head];
  const bool append = a.k_new != nullptr;
  const bool can_append = append && old_len < a.cap;
  if (append && !can_append && split == 0 && threadIdx.x == 0) atomicOr(a.flag, 1);
  const int eff_len = can_append ? old_len + 1 : old_len;
  const T* k_new = append ? reinterpret_cast<const T*>(a.k_new) + (size_t)head * D : nullptr;
  const T* v_new = append ? reinterpret_cast<const T*>(a.v_new) + (size_t)head * D : nullptr;

  // Append: the workgroup whose slice holds row old_len writes it to the cache.  Nobody
  // reads that row from the cache in this launch (the new token is read from k_new).
  if (can_append && min(old_len / a.split_len, a.nsplit - 1) == split) {
    for (int e = threadIdx.x; e < D; e += blockDim.x) {
      k_cache[cache_off + (size_t)old_len * D + e] = k_new[e];
      v_cache[cache_off + (size_t)old_len * D + e] = v_new[e];
    }
  }

  int t0 = split * a.split_len;
  const int t1 = (split == a.nsplit - 1) ? eff_len : min(t0 + a.split_len, eff_len);
  if (t0 > t1) t0 = t1;

  // Query fragments (A operand): row m = query g (zero beyond G), 8 dims per lane.
  FragT qf[KS];
  {
    const int g = lane & 15;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = (g < G) ? load_frag(qh + (size_t)g * D + 32 * ks + 8 * (lane >> 4)) : zero_frag<T>();
  }
  const float c2 = a.scale * kLog2e;

  // Token blocks of TB = 32 rows; wave w takes blocks w, w+4, ...
  //  * K rows are MFMA B fragments of Q.K^T (lane: row (lane%16) + 16h, 8 dims at
  //    8*(lane/16) + 32*ks);
  //  * V rows are loaded as token pairs (lane: rows 2p, 2p+1 with p = lane%16, 8-column
  //    groups lane/16 + 4c) and written transposed to the wave's LDS tile, each dword
  //    holding the two tokens of one column;
  //  * P goes to LDS as the A operand of P.V (bf16 for bf16 caches, fp32 otherwise) and
  //    P.V runs on MFMA: out[g][dim] in the same lane layout as the logits, so the online
  //    softmax rescale needs no shuffles.
  // The next block's rows are requested once the current ones have left the registers.
  FragT kf[2][KS], vf[2][NVC];
  auto load_block = [&](int j0) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int j = j0 + 16 * hh + (lane & 15);
      const T* row = (j == old_len && can_append) ? k_new : kc + (size_t)j * D;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kf[hh][ks] = (j < t1) ? load_frag(row + 32 * ks + 8 * (lane >> 4)) : zero_frag<T>();
    }
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int j = j0 + 2 * (lane & 15) + hh;
      const T* row = (j == old_len && can_append) ? v_new : vc + (size_t)j * D;
#pragma unroll
      for (int c = 0; c < NVC; ++c)
        vf[hh][c] = (j < t1) ? load_frag(row + 8 * ((lane >> 4) + 4 * c)) : zero_frag<T>();
    }
  };
  const int nblk = (t1 - t0 + TB - 1) / TB;
  if (wave < nblk) load_block(t0 + TB * wave);

  // ---- rows of S_tilde q for this slice (all rows when fused)
  const int ne = a.n_e[head];
  const float inv_n = ne > 0 ? 1.f / (float)ne : 0.f;
  if (ne > 0 && a.order >= 1) {
    const int rs = (D + a.nsplit - 1) / a.nsplit;
    const int r0 = split * rs, r1 = min(D, r0 + rs);
    float* dst = FUSED ? &s_sq[0][0] : a.sq + (size_t)head * G * D;
    stilde_q<T, D>(a, head, qh, G, r0, r1, wave, lane, inv_n, dst);
  }

  float m_run[4], l_run[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { m_run[i] = -INFINITY; l_run[i] = 0.f; }
  f32x4 oacc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) oacc[nt] = zero4();
  T (*vt)[TB + PT] = s_vt[wave];
  T (*sp)[TB + PT] = s_p[wave];
  const int gbase = 4 * (lane >> 4);

  for (int blk = wave; blk < nblk; blk += 4) {
    const int j0 = t0 + TB * blk;
    // ---- logits for the two 16-token halves
    f32x4 acc[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      acc[hh] = zero4();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) mma(acc[hh], qf[ks], kf[hh][ks]);
    }
    // ---- V^T into the wave's LDS tile (columns 2p, 2p+1 of row dim)
    {
      const int p2 = 2 * (lane & 15);
#pragma unroll
      for (int c = 0; c < NVC; ++c) {
        const int col0 = 8 * ((lane >> 4) + 4 * c);
        if constexpr (sizeof(T) == 2) {
          const u32x4_t w0 = __builtin_bit_cast(u32x4_t, vf[0][c]);
          const u32x4_t w1 = __builtin_bit_cast(u32x4_t, vf[1][c]);
#pragma unroll
          for (int w = 0; w < 4; ++w)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
              store_vpair(reinterpret_cast<bf16_t*>(&vt[col0 + 2 * w + hh][p2]), w0[w], w1[w], hh);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            *reinterpret_cast<float2*>(&vt[col0 + e][p2]) = make_float2(elem_f(vf[0][c], e), elem_f(vf[1][c], e));
        }
      }
    }
    if (blk + 4 < nblk) load_block(j0 + 4 * TB);
    // ---- online softmax over the 32 tokens (rows g = gbase + i)
    float alpha[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ja = j0 + (lane & 15), jb = ja + 16;
      const bool gok = gbase + i < G;
      const float xa = (ja < t1 && gok) ? acc[0][i] * c2 : -INFINITY;
      const float xb = (jb < t1 && gok) ? acc[1][i] * c2 : -INFINITY;
      const float bm = row16_max(fmaxf(xa, xb));
      const float mn = fmaxf(m_run[i], bm);
      float pa = 0.f, pb = 0.f;
      if (mn == -INFINITY) {
        alpha[i] = 1.f;
      } else {
        alpha[i] = fast_exp2(m_run[i] - mn);
        pa = fast_exp2(xa - mn);
        pb = fast_exp2(xb - mn);
      }
      l_run[i] = l_run[i] * alpha[i] + row16_sum(pa + pb);
      m_run[i] = mn;
      if (gbase + i < GMAX) {
        sp[gbase + i][lane & 15] = from_f<T>(pa);
        sp[gbase + i][16 + (lane & 15)] = from_f<T>(pb);
      }
    }
    // ---- O = alpha * O + P . V on MFMA (A = P rows g, B = V^T)
    const FragT pfr = ((lane & 15) < G) ? load_frag(&sp[lane & 15][8 * (lane >> 4)]) : zero_frag<T>();
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) oacc[nt][i] *= alpha[i];
      mma(oacc[nt], pfr, load_frag(&vt[16 * nt + (lane & 15)][8 * (lane >> 4)]));
    }
  }

  // ---- per-wave results to LDS: lane holds out[g = gbase + i][16*nt + lane%16]
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (gbase + i < GMAX) s_o[wave][gbase + i][16 * nt + (lane & 15)] = oacc[nt][i];
  if ((lane & 15) == 0) {
    const int gb = 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (gb + i < GMAX) { s_m[wave][gb + i] = m_run[i]; s_l[wave][gb + i] = l_run[i]; }
  }
  __syncthreads();

  if constexpr (!FUSED) {
    const size_t pbase = ((size_t)head * a.nsplit + split) * G;
    for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
      const int g = idx / D, e = idx % D;
      float M = -INFINITY;
      for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][g]);
      float acc = 0.f;
      if (M != -INFINITY)
        for (int w = 0; w < 4; ++w) acc += s_o[w][g][e] * fast_exp2(s_m[w][g] - M);
      a.part_o[(pbase + g) * D + e] = acc;
    }
    for (int g = threadIdx.x; g < G; g += blockDim.x) {
      float M = -INFINITY;
      for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][g]);
      float l = 0.f;
      if (M != -INFINITY)
        for (int w = 0; w < 4; ++w) l += s_l[w][g] * fast_exp2(s_m[w][g] - M);
      a.part_ml[(pbase + g) * 2 + 0] = M;
      a.part_ml[(pbase + g) * 2 + 1] = l;
    }
  } else {
    // a single slice: merge the waves and apply the correction here (one wave per query)
    for (int g = wave; g < G; g += 4) {
      float M = -INFINITY;
      for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][g]);
      float l = 0.f;
      if (M != -INFINITY)
        for (int w = 0; w < 4; ++w) l += s_l[w][g] * fast_exp2(s_m[w][g] - M);
      float dot = 0.f;
      if (ne > 0) {
        for (int e = lane; e < D; e += 64) dot += to_f(qh[(size_t)g * D + e]) * a.s_k[(size_t)head * D + e];
        dot = wave_sum(dot);
      }
      const Mix mx = mix_weights(M, l, ne, dot, a.scale);
      const size_t pair = (size_t)head * G + g;
      if (lane == 0) {
        if (a.lse_out) a.lse_out[pair] = mx.log_zr;
        if (a.w_r_out) a.w_r_out[pair] = mx.w_r;
      }
      T* out = reinterpret_cast<T*>(a.out) + pair * D;
      for (int e = lane; e < D; e += 64) {
        float num = 0.f;
        if (M != -INFINITY)
          for (int w = 0; w < 4; ++w) num += s_o[w][g][e] * fast_exp2(s_m[w][g] - M);
        const float f_r = l > 0.f ? num / l : 0.f;
        float res = f_r;
        if (ne > 0) {
          float fe = a.s_v[(size_t)head * D + e] * inv_n;
          if (a.order >= 1) fe += a.scale * inv_n * s_sq[g][e];
          res = mx.w_r * f_r + (1.f - mx.w_r) * fe;
        }
        out[e] = from_f<T>(res);
      }
    }
    if (threadIdx.x == 0 && can_append) a.lens[head] = old_len + 1;
  }
}

// Merge of one query head's slices and the moment correction (one wave).
template <class T, int D>
__device__ void decode_merge_query(const DecodeArgs& a, int bh, int g, int lane) {
  constexpr int CPL = D / 64;
  const int G = a.G;
  const int pair = bh * G + g;             // (b, hq) flattened
  const T* q = reinterpret_cast<const T*>(a.q) + (size_t)pair * D;
  T* out = reinterpret_cast<T*>(a.out);

  float M = -INFINITY;
  for (int s = 0; s < a.nsplit; ++s) M = fmaxf(M, a.part_ml[(((size_t)bh * a.nsplit + s) * G + g) * 2]);
  float l = 0.f, o[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) o[c] = 0.f;
  if (M != -INFINITY) {
    for (int s = 0; s < a.nsplit; ++s) {
      const size_t pb = ((size_t)bh * a.nsplit + s) * G + g;
      const float w = fast_exp2(a.part_ml[pb * 2] - M);
      l += a.part_ml[pb * 2 + 1] * w;
#pragma unroll
      for (int c = 0; c < CPL; ++c) o[c] += a.part_o[pb * D + lane * CPL + c] * w;
    }
  }
  const int ne = a.n_e[bh];
  float dot = 0.f;
  if (ne > 0) {
#pragma unroll
    for (int c = 0; c < CPL; ++c) dot += to_f(q[lane * CPL + c]) * a.s_k[(size_t)bh * D + lane * CPL + c];
    dot = wave_sum(dot);
  }
  const Mix mx = mix_weights(M, l, ne, dot, a.scale);
  const float inv_n = ne > 0 ? 1.f / (float)ne : 0.f;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int e = lane * CPL + c;
    const float f_r = (l > 0.f) ? o[c] / l : 0.f;
    float res = f_r;
    if (ne > 0) {
      float fe = a.s_v[(size_t)bh * D + e] * inv_n;
      if (a.order >= 1) fe += a.scale * inv_n * a.sq[((size_t)bh * G + g) * D + e];
      res = mx.w_r * f_r + (1.f - mx.w_r) * fe;
    }
    out[(size_t)pair * D + e] = from_f<T>(res);
  }
  if (lane == 0) {
    if (a.lse_out) a.lse_out[pair] = mx.log_zr;
    if (a.w_r_out) a.w_r_out[pair] = mx.w_r;
  }
}

// Merge kernel: one wave per (b, query head); the g == 0 wave of a KV head also bumps
// lens after an append (every slice workgroup read lens in the previous launch).
template <class T, int D>
__global__ void __launch_bounds__(256) k_decode_merge(DecodeArgs a) {
  const int lane = threadIdx.x & 63;
  const int pair = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (pair >= a.n_pairs) return;
  const int bh = pair / a.G, g = pair % a.G;
  decode_merge_query<T, D>(a, bh, g, lane);
  if (g == 0 && lane == 0 && a.k_new != nullptr && a.lens[bh] < a.cap) a.lens[bh] += 1;
}

template <class T, int D, int GMAX>
static hipError_t launch_decode_t(const DecodeArgs& a, hipStream_t st) {
  if (a.nsplit == 1) {
    hipLaunchKernelGGL((k_decode<T, D, GMAX, true>), dim3(1, a.n_heads), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((k_decode<T, D, GMAX, false>), dim3(a.nsplit, a.n_heads), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_decode_merge<T, D>), dim3((a.n_pairs + 3) / 4), dim3(256), 0, st, a);
  return hipGetLastError();
}

template <class T, int D>
static hipError_t launch_decode_g(const DecodeArgs& a, hipStream_t st) {
  if (a.G <= 4) return launch_decode_t<T, D, 4>(a, st);
  if (a.G <= 8) return launch_decode_t<T, D, 8>(a, st);
  return launch_decode_t<T, D, 16>(a, st);
}

hipError_t launch_decode(const DecodeArgs& a, bool bf16, int d, hipStream_t st) {
  if (bf16) return d == 64 ? launch_decode_g<bf16_t, 64>(a, st) : launch_decode_g<bf16_t, 128>(a, st);
  return d == 64 ? launch_decode_g<float, 64>(a, st) : launch_decode_g<float, 128>(a, st);
}

}  // namespace mkv
