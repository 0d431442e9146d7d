// Corrected decode attention over the retained cache (Algorithm 1 Phase 2; Eqs. fhat,
// jensen and fused; log-domain mixing weight of App. C.2), split-K over the cache.
//
// One kernel, grid (nsplit, B*Hkv), 256 threads.  Each workgroup streams one slice of one
// KV head's retained rows for all G query heads of the group: Q.K^T on MFMA (the G
// queries padded to 16 rows), online softmax in the base-2 domain, P.V on the vector ALU
// over coalesced rows.  It also computes its share of the rows of S_tilde q (clamped
// covariance times each query), so the d x d summary is read once per head in total.
// The new token (if any) is appended by the workgroup owning its row.  The last
// workgroup of a head to finish (a per-head arrival counter in the workspace) merges the
// slices in a fixed order (f_R, log Z_R), mixes in the first-order estimate f_E_hat with
// the Jensen weight, writes the outputs, bumps lens and resets the counter.
#include "mkv_device.h"
#include "mkv_launch.h"

namespace mkv {

template <class T, int D>
__device__ void decode_merge_query(const DecodeArgs& a, int bh, int g, int lane);

template <class T, int D, int GMAX>
__global__ void __launch_bounds__(256) k_decode(DecodeArgs a) {
  constexpr int KS = D / 32;        // MFMA contraction steps per row
  constexpr int LPR = D / 8;        // lanes per row in the coalesced V layout
  constexpr int TPL = 64 / LPR;     // rows per wave-wide V load
  constexpr int NG4 = (GMAX + 3) / 4;  // 16-lane rows of the MFMA output holding queries
  static_assert(GMAX <= 16, "G <= 16");

  __shared__ float s_o[4][GMAX][D];
  __shared__ float s_m[4][GMAX];
  __shared__ float s_l[4][GMAX];

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
  if (can_append) {
    int owner = min(old_len / a.split_len, a.nsplit - 1);
    if (owner == split) {
      for (int e = threadIdx.x; e < D; e += blockDim.x) {
        k_cache[cache_off + (size_t)old_len * D + e] = k_new[e];
        v_cache[cache_off + (size_t)old_len * D + e] = v_new[e];
      }
    }
  }

  int t0 = split * a.split_len;
  int t1 = (split == a.nsplit - 1) ? eff_len : min(t0 + a.split_len, eff_len);
  if (t0 > t1) t0 = t1;

  // Query fragments (A operand): row m = query g (zero beyond G), 8 dims per lane.
  typename Frag<T>::type qf[KS];
  {
    const int g = lane & 15;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = (g < G) ? load_frag(qh + (size_t)g * D + 32 * ks + 8 * (lane >> 4)) : zero_frag<T>();
  }
  const float c2 = a.scale * kLog2e;

  float m_run[4], l_run[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { m_run[i] = -INFINITY; l_run[i] = 0.f; }
  float o[GMAX][8];
#pragma unroll
  for (int g = 0; g < GMAX; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;

  const int nblk = (t1 - t0 + 15) >> 4;
  for (int blk = wave; blk < nblk; blk += 4) {
    const int j0 = t0 + 16 * blk;
    // ---- logits: lane holds s[g = 4*(lane/16) + i][token j0 + lane%16]
    f32x4 acc = zero4();
    {
      const int j = j0 + (lane & 15);
      const T* row = (j == old_len && can_append) ? k_new : kc + (size_t)j * D;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        typename Frag<T>::type bf = (j < t1) ? load_frag(row + 32 * ks + 8 * (lane >> 4)) : zero_frag<T>();
        mma(acc, qf[ks], bf);
      }
    }
    float p[4], alpha[4];
    {
      const int j = j0 + (lane & 15);
      const int gbase = 4 * (lane >> 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float s2 = (j < t1 && gbase + i < G) ? acc[i] * c2 : -INFINITY;
        float bm = row16_max(s2);
        float mn = fmaxf(m_run[i], bm);
        if (mn == -INFINITY) {
          alpha[i] = 1.f;
          p[i] = 0.f;
        } else {
          alpha[i] = fast_exp2(m_run[i] - mn);
          p[i] = fast_exp2(s2 - mn);
        }
        l_run[i] = l_run[i] * alpha[i] + row16_sum(p[i]);
        m_run[i] = mn;
      }
    }
    // ---- P.V: lane covers dims 8*(lane%LPR).. of rows j0 + lane/LPR + TPL*u
#pragma unroll
    for (int g = 0; g < GMAX; ++g) {
      if (g < G) {
        float al = __shfl(alpha[g & 3], 16 * (g >> 2));
#pragma unroll
        for (int e = 0; e < 8; ++e) o[g][e] *= al;
      }
    }
#pragma unroll
    for (int u = 0; u < 16 / TPL; ++u) {
      const int tl = lane / LPR + TPL * u;  // token within the block
      const int j = j0 + tl;
      float v[8];
      if (j < t1) {
        const T* row = (j == old_len && can_append) ? v_new : vc + (size_t)j * D;
        typename Frag<T>::type vf = load_frag(row + 8 * (lane % LPR));
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = elem_f(vf, e);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;
      }
#pragma unroll
      for (int g = 0; g < GMAX; ++g) {
        float pg = __shfl(p[g & 3], 16 * (g >> 2) + tl);
        if (g < G) {
#pragma unroll
          for (int e = 0; e < 8; ++e) o[g][e] += pg * v[e];
        }
      }
    }
  }

  // ---- reduce o over the lanes sharing dims, then over the waves (fixed order)
#pragma unroll
  for (int g = 0; g < GMAX; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float x = o[g][e];
      if (LPR == 8) x += __shfl_xor(x, 8);
      x = cross_row_sum(x);
      o[g][e] = x;
    }
  if (lane < LPR) {
#pragma unroll
    for (int g = 0; g < GMAX; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) s_o[wave][g][8 * lane + e] = o[g][e];
  }
  if ((lane & 15) == 0) {
    const int gb = 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (gb + i < GMAX) { s_m[wave][gb + i] = m_run[i]; s_l[wave][gb + i] = l_run[i]; }
  }
  __syncthreads();
  {
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
  }

  // ---- this slice's rows of S_tilde q for every query of the group
  const int ne = a.n_e[head];
  if (ne > 0 && a.order >= 1) {
    const int rs = (D + a.nsplit - 1) / a.nsplit;
    const int r0 = split * rs, r1 = min(D, r0 + rs);
    const float inv_n = 1.f / (float)ne;
    const float* Sh = a.S + (size_t)head * D * D;
    const float* skh = a.s_k + (size_t)head * D;
    const float* svh = a.s_v + (size_t)head * D;
    constexpr int CPL = D / 64;  // columns per lane
    float qc[GMAX][CPL], skc[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      skc[c] = skh[lane * CPL + c];
#pragma unroll
      for (int g = 0; g < GMAX; ++g) qc[g][c] = (g < G) ? to_f(qh[(size_t)g * D + lane * CPL + c]) : 0.f;
    }
    for (int r = r0 + wave; r < r1; r += 4) {
      const float sv = svh[r];
      float part[GMAX];
#pragma unroll
      for (int g = 0; g < GMAX; ++g) part[g] = 0.f;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        float st = Sh[(size_t)r * D + lane * CPL + c] - sv * skc[c] * inv_n;
        if (fabsf(st) < a.tau) st = 0.f;
#pragma unroll
        for (int g = 0; g < GMAX; ++g) part[g] += st * qc[g][c];
      }
#pragma unroll
      for (int g = 0; g < GMAX; ++g) {
        float t = wave_sum(part[g]);
        if (g < G && lane == 0) a.sq[((size_t)head * G + g) * D + r] = t;
      }
    }
  }

  // ---- arrival: the last workgroup of this head merges (release by every thread,
  // then one counter increment; acquire before reading the other slices)
  __shared__ int s_last;
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(a.counter + head, 1) == a.nsplit - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  for (int g = wave; g < G; g += 4) decode_merge_query<T, D>(a, head, g, lane);
  if (threadIdx.x == 0) {
    a.counter[head] = 0;
    if (can_append) a.lens[head] = old_len + 1;
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
  const float log_zr = (l > 0.f) ? (M + __log2f(l)) * kLn2 : -INFINITY;
  float f_r[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) f_r[c] = (l > 0.f) ? o[c] / l : 0.f;

  const int ne = a.n_e[bh];
  float w_r = 1.f;
  float res[CPL];
  if (ne == 0) {
#pragma unroll
    for (int c = 0; c < CPL; ++c) res[c] = f_r[c];
  } else {
    const float inv_n = 1.f / (float)ne;
    float dot = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) dot += to_f(q[lane * CPL + c]) * a.s_k[(size_t)bh * D + lane * CPL + c];
    dot = wave_sum(dot);
    const float log_ze = logf((float)ne) + a.scale * dot * inv_n;   // Jensen estimate
    const float hi = fmaxf(log_zr, log_ze);
    const float lse = hi + logf(expf(log_zr - hi) + expf(log_ze - hi));
    w_r = expf(log_zr - lse);
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int e = lane * CPL + c;
      float fe = a.s_v[(size_t)bh * D + e] * inv_n;
      if (a.order >= 1) fe += a.scale * inv_n * a.sq[((size_t)bh * G + g) * D + e];
      res[c] = w_r * f_r[c] + (1.f - w_r) * fe;
    }
  }
#pragma unroll
  for (int c = 0; c < CPL; ++c) out[(size_t)pair * D + lane * CPL + c] = from_f<T>(res[c]);
  if (lane == 0) {
    if (a.lse_out) a.lse_out[pair] = log_zr;
    if (a.w_r_out) a.w_r_out[pair] = w_r;
  }
}

template <class T, int D, int GMAX>
static hipError_t launch_decode_t(const DecodeArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((k_decode<T, D, GMAX>), dim3(a.nsplit, a.n_heads), dim3(256), 0, st, a);
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
