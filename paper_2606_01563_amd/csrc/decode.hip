// Corrected decode attention over the retained cache (Algorithm 1 Phase 2; Eqs. fhat,
// jensen and fused; log-domain mixing weight of App. C.2).
//
// Two launch shapes, chosen by the host from the cache length bound:
//
// fused   k_decode_fused: one 4-wave workgroup per KV head, one launch.  Wave w computes
//         rows [32w, 32w + 32) of S_tilde q (S_tilde = S - s_v s_k^T / n_e, clamped; formed
//         from the raw S as it is loaded, or read in the prepared form) and attends to the
//         32-row blocks w, w + 4, ... of the retained cache for all G query heads of the
//         group; the four partial softmax states are merged
//         in LDS, the new token is folded in, and the moment correction is applied.  The
//         S rows and the first cache block are requested together, so the S_tilde q
//         products run while the cache rows are in flight.  Used for short caches, where
//         a decode call is latency bound.
//
// split   k_decode_slice: one launch, a 1-D grid of n_heads x (nsq + nsplit) single-wave
//         workgroups:
//         * n_heads x nsq waves of 32 rows of S_tilde q;
//         * n_heads x nsplit token slices (split_len rows below lens) of one KV head,
//           each an unnormalised (o, max, sum) partial;
//         each wave hands its result over through agent-scope stores and counts itself in
//         on the head's counter, and the wave that completes the count merges the head:
//         per query, the slices in a fixed order, then the new token, then the
//         correction (so the result does not depend on which wave merges).
//         Used for long caches: reading is bound by how much each CU keeps in flight, so
//         the finishing time is set by the busiest CU, and thousands of short slices let
//         the dispatcher balance a few hundred heads over 256 CUs.
//
// Common to both: Q.K^T and P.V run on MFMA over 32-token blocks (the G queries padded to
// 16 rows) with the online softmax in the base-2 domain.  The new token (k_new, v_new) is
// written to row lens of the cache by the wave whose range holds that row and is attended
// to from k_new / v_new, so no cache read depends on the append.
#include "mkv_device.h"
#include "mkv_decode.h"

namespace mkv {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Length of one KV head's retained set for this call.  lens is clamped so that a
// corrupt value can never move a read or the append outside the cache.
struct HeadLen {
  int old_len;      // lens before the append
  bool can_append;  // a new token is given and its row is inside the cache
  int cache_len;    // cache rows attended to: old_len clamped to [0, cap]
};
__device__ __forceinline__ HeadLen head_len(const DecodeArgs& a, int old_len) {
  HeadLen r;
  r.old_len = old_len;
  r.can_append = a.k_new != nullptr && old_len >= 0 && old_len < a.cap;
  r.cache_len = min(max(old_len, 0), a.cap);
  return r;
}
__device__ __forceinline__ int live_slices(const DecodeArgs& a, int cache_len) {
  return min(a.nsplit, (cache_len + a.split_len - 1) / a.split_len);
}

// Orders the wave's own LDS writes and reads for the compiler.  A wave's LDS operations
// are carried out in issue order, so lanes of one wave exchanging data through LDS need
// no hardware wait beyond that.
__device__ __forceinline__ void wave_lds_order() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// ---------------------------------------------------------------- in-launch hand-off
// Partial results that one workgroup hands to another within the split launch go through
// agent-scope relaxed atomic stores and loads, which are not served from the per-XCD
// caches (those are not kept coherent with each other).  A writer waits until its own
// stores have completed before it counts itself in on the head's arrival counter, and the
// last arrival reads the partials only after the count, so no device-scope fence is
// needed (on this part such a fence writes back and invalidates a whole L2).
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), __float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent2(float* p, float x, float y) {
  const uint64_t u = (uint64_t)__float_as_uint(x) | ((uint64_t)__float_as_uint(y) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_agent2(const float* p) {
  const uint64_t u = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)u), __uint_as_float((uint32_t)(u >> 32)));
}
// s_waitcnt with vmcnt = 0 and the other counters at their maximum: every vector memory
// operation of the wave issued so far (stores included) has completed.
constexpr int kWaitVmem = 0x0F70;
__device__ __forceinline__ void stores_complete() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_waitcnt(kWaitVmem);
}
__device__ __forceinline__ void loads_after_count() {
  __builtin_amdgcn_s_waitcnt(kWaitVmem);
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Query fragments of one KV head's group (A operand of Q.K^T, B operand of S_tilde q):
// lane l holds 8 dims at 32 ks + 8 (l / 16) of query l % 16; queries past G are zero.
template <class T, int D>
__device__ __forceinline__ void load_query_frags(const T* qh, int G, int lane,
                                                 typename Frag<T>::type (&qf)[D / 32]) {
  const int g = lane & 15, gc = min(g, G - 1);
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    const typename Frag<T>::type f = load_frag(qh + (size_t)gc * D + 32 * ks + 8 * (lane >> 4));
    qf[ks] = g < G ? f : zero_frag<T>();
  }
}

// The new token: the wave given the job copies k_new / v_new to cache row `row`, 16 bytes
// per lane (loads first, then stores).
template <class T, int D>
__device__ __forceinline__ void append_row(const DecodeArgs& a, int head, int row, int lane) {
  constexpr int NV = D * (int)sizeof(T) / 16;  // 16-byte pieces of a row
  if (lane < 2 * NV) {
    const bool is_v = lane >= NV;
    const int piece = lane % NV;
    const uint4* src = reinterpret_cast<const uint4*>(
        reinterpret_cast<const T*>(is_v ? a.v_new : a.k_new) + (size_t)head * D) + piece;
    T* cache = reinterpret_cast<T*>(is_v ? a.v_cache : a.k_cache);
    uint4* dst = reinterpret_cast<uint4*>(cache + ((size_t)head * a.cap + row) * D) + piece;
    *dst = *src;
  }
}

// ---------------------------------------------------------------- S_tilde q
// Rows [r0, r0 + 32) of S_tilde q (unscaled) for the queries held in the query fragments
// (query g in MFMA column g).  load() issues every read; compute() writes result (g, r) to
// dst[g * D + r] for g < G.  Four forms of the summary:
//  * raw S (PREP = false): fp32 MFMA; S_tilde = S - s_v s_k^T / n_e, clamped at tau, is
//    formed as the rows are loaded;
//  * prepared, fp32 caches: the stored S_tilde on fp32 MFMA;
//  * prepared, bf16 caches: the stored hi / lo bf16 planes on bf16 MFMA, two products per
//    32-wide step against the (exact) bf16 queries;
//  * prepared in half precision (PREP = 2, bf16 caches): the hi plane alone, one product;
//  * raw S stored in bf16 (PREP = 3): as the raw fp32 form, from bf16 loads.
template <class T, int D, int PREP>
struct SqRows {
  static constexpr int KS = D / 32;
  static constexpr bool HILO = PREP == 1 && sizeof(T) == 2;
  static constexpr bool HI1 = PREP == 2;  // one bf16 plane (bf16 caches only)
  static constexpr bool RAW = PREP == 0 || PREP == 3;  // centred and clamped here
  f32x8 raw[2][KS];
  bf16x8 hi[2][KS], lo[2][KS];
  f32x8 skc[KS];
  float sv[2];
  int ne;

  __device__ __forceinline__ void load(const DecodeArgs& a, int head, int r0, int lane) {
    const int col = 8 * (lane >> 4);
    if constexpr (HILO) {
      const bf16_t* P = reinterpret_cast<const bf16_t*>(a.S) + (size_t)head * 2 * D * D;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int row = r0 + 16 * u + (lane & 15);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          hi[u][ks] = load_frag(P + (size_t)row * D + 32 * ks + col);
          lo[u][ks] = load_frag(P + (size_t)(D + row) * D + 32 * ks + col);
        }
      }
    } else if constexpr (HI1) {
      const bf16_t* P = reinterpret_cast<const bf16_t*>(a.S) + (size_t)head * D * D;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int row = r0 + 16 * u + (lane & 15);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) hi[u][ks] = load_frag(P + (size_t)row * D + 32 * ks + col);
      }
    } else {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int row = r0 + 16 * u + (lane & 15);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const size_t off = ((size_t)head * D + row) * D + 32 * ks + col;
          if constexpr (PREP == 3) {
            const bf16x8 b = load_frag(reinterpret_cast<const bf16_t*>(a.S) + off);
#pragma unroll
            for (int e = 0; e < 8; ++e) raw[u][ks][e] = elem_f(b, e);
          } else {
            raw[u][ks] = load_frag(a.S + off);
          }
        }
        if constexpr (RAW) sv[u] = a.s_v[(size_t)head * D + row];
      }
      if constexpr (RAW) {
        ne = a.n_e[head];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) skc[ks] = load_frag(a.s_k + (size_t)head * D + 32 * ks + col);
      }
    }
  }

  // AGENT: dst is read by another workgroup of the launch (agent-scope stores)
  template <bool AGENT = false>
  __device__ __forceinline__ void compute(const DecodeArgs& a, const typename Frag<T>::type (&qf)[KS],
                                          int r0, int lane, float* dst) {
    const int g = lane & 15;
    f32x4 acc[2];
    if constexpr (HILO) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        acc[u] = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          mma(acc[u], hi[u][ks], qf[ks]);
          mma(acc[u], lo[u][ks], qf[ks]);
        }
      }
    } else if constexpr (HI1) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        acc[u] = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) mma(acc[u], hi[u][ks], qf[ks]);
      }
    } else {
      float inv_n = 0.f;
      if constexpr (RAW) inv_n = ne > 0 ? 1.f / (float)ne : 0.f;
      f32x8 qb[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) qb[ks][e] = elem_f(qf[ks], e);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        acc[u] = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          f32x8 af;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            if constexpr (PREP == 1) {
              af[e] = raw[u][ks][e];
            } else {
              const float st = raw[u][ks][e] - sv[u] * (skc[ks][e] * inv_n);
              af[e] = fabsf(st) < a.tau ? 0.f : st;
            }
          }
          mma(acc[u], af, qb[ks]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int i = 0; i < 4; i += 2) {
        float* p = dst + (size_t)g * D + r0 + 16 * u + 4 * (lane >> 4) + i;
        if (g < a.G) {
          if constexpr (AGENT) {
            st_agent2(p, acc[u][i], acc[u][i + 1]);
          } else {
            p[0] = acc[u][i];
            p[1] = acc[u][i + 1];
          }
        }
      }
  }
};

// Decode form of the summary: S_tilde = S - s_v s_k^T / n_e with entries below tau set to
// zero, computed with the same fp32 arithmetic as the raw-summary decode path, stored as
// hi = RNE_bf16(S_tilde) and lo = RNE_bf16(S_tilde - hi) planes for bf16 caches (the hi
// plane alone for the half-precision form, hi_only), or as fp32.
// Grid (D * D / 8 / 256, n_heads); a thread handles 8 consecutive entries of one row.
template <class T, int D>
__global__ void __launch_bounds__(256) k_prepare_summary(DecodeArgs a, void* prepared, int hi_only) {
  const int head = blockIdx.y;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= D * D / 8) return;
  const int row = idx / (D / 8), c0 = 8 * (idx % (D / 8));
  const int ne = a.n_e[head];
  const float inv_n = ne > 0 ? 1.f / (float)ne : 0.f;
  const f32x8 raw = load_frag(a.S + ((size_t)head * D + row) * D + c0);
  const f32x8 skc = load_frag(a.s_k + (size_t)head * D + c0);
  const float sv = a.s_v[(size_t)head * D + row];
  float st[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float t = raw[e] - sv * (skc[e] * inv_n);
    st[e] = (ne <= 0 || fabsf(t) < a.tau) ? 0.f : t;
  }
  if constexpr (sizeof(T) == 2) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const bf16_t h0 = f2bf(st[e]), h1 = f2bf(st[e + 1]);
      const bf16_t l0 = f2bf(st[e] - bf2f(h0)), l1 = f2bf(st[e + 1] - bf2f(h1));
      h[e / 2] = (uint32_t)h0 | ((uint32_t)h1 << 16);
      l[e / 2] = (uint32_t)l0 | ((uint32_t)l1 << 16);
    }
    bf16_t* P = reinterpret_cast<bf16_t*>(prepared) + (size_t)head * (hi_only ? 1 : 2) * D * D;
    *reinterpret_cast<uint4*>(P + (size_t)row * D + c0) = make_uint4(h[0], h[1], h[2], h[3]);
    if (!hi_only)
      *reinterpret_cast<uint4*>(P + (size_t)(D + row) * D + c0) = make_uint4(l[0], l[1], l[2], l[3]);
  } else {
    float4* P = reinterpret_cast<float4*>(reinterpret_cast<float*>(prepared) + ((size_t)head * D + row) * D + c0);
    P[0] = make_float4(st[0], st[1], st[2], st[3]);
    P[1] = make_float4(st[4], st[5], st[6], st[7]);
  }
}

// ---------------------------------------------------------------- block attention
// One wave's online-softmax attention over 32-row blocks of one KV head's cache rows
// below t_end, for the G queries of the group:
//  * K rows are MFMA B fragments of Q.K^T (lane: row (lane%16) + 16h, 8 dims at
//    8*(lane/16) + 32*ks);
//  * V rows are loaded as token pairs (lane: rows 2p, 2p+1 with p = lane%16, 8-column
//    groups lane/16 + 4c) and written to the wave's LDS tile as they are (bf16; read back
//    as B fragments of P.V with the transposing LDS read) or transposed (fp32, each
//    64-bit word holding the two tokens of one column);
//  * P goes to LDS as the A operand of P.V (bf16 for bf16 caches, fp32 otherwise) and P.V
//    runs on MFMA: out[g][dim] in the same lane layout as the logits, so the online
//    softmax rescale needs no shuffles.
// The next block's rows are requested once the current ones have left the registers.
// Lane l ends with rows g = 4 (l / 16) + i: (m_run[i], l_run[i]) in log2 units and
// o[g][16 nt + l % 16] = oacc[nt][i].
template <class T, int D, int GMAX>
struct BlockAttn {
  static constexpr int KS = D / 32;        // MFMA contraction steps per row
  static constexpr int TB = 32;            // tokens per block
  static constexpr int NVC = D / 32;       // V chunks (16 or 32 bytes) per lane and token
  static constexpr int NT = D / 16;        // 16-column output tiles of P.V
  static constexpr int PT = 16 / (int)sizeof(T);  // LDS row padding (16 bytes)
  static constexpr bool TR = sizeof(T) == 2;       // bf16: V kept in its own layout
  static constexpr int LDV = D + 16;               // bf16 V rows padded by 32 bytes
  typedef typename Frag<T>::type FragT;
  // bf16: the block's V rows as they are, read back transposed as MFMA operands; fp32:
  // V^T, written transposed
  typedef typename Pick<TR, T[TB][LDV], T[D][TB + PT]>::type VtTile;
  typedef T PTile[16][TB + PT];

  const T* kc;
  const T* vc;
  int t_end;
  FragT kf[2][KS], vf[2][NVC];
  float m_run[4], l_run[4];
  f32x4 oacc[NT];

  // Rows at or past t_end are loaded from row t_end - 1 (row 0 when t_end = 0), so no
  // load sits under a per-lane condition: their logits are masked in run() and their
  // weights are zero, so the copies contribute nothing.
  __device__ __forceinline__ void load(int j0, int lane) {
    const int last = max(t_end, 1) - 1;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int j = min(j0 + 16 * hh + (lane & 15), last);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kf[hh][ks] = load_frag(kc + (size_t)j * D + 32 * ks + 8 * (lane >> 4));
    }
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int j = min(j0 + 2 * (lane & 15) + hh, last);
#pragma unroll
      for (int c = 0; c < NVC; ++c)
        vf[hh][c] = load_frag(vc + (size_t)j * D + 8 * ((lane >> 4) + 4 * c));
    }
  }

  // V rows of the block at j0 at or past t_end to zero (K rows there only feed masked logits)
  __device__ __forceinline__ void clear_v_past_end(int j0, int lane) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const bool ok = j0 + 2 * (lane & 15) + hh < t_end;
#pragma unroll
      for (int c = 0; c < NVC; ++c) vf[hh][c] = ok ? vf[hh][c] : zero_frag<T>();
    }
  }

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < 4; ++i) { m_run[i] = -INFINITY; l_run[i] = 0.f; }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) oacc[nt] = zero4();
  }

  // Blocks at j_first, j_first + stride, ... below t_end; load(j_first) was issued.
  __device__ __forceinline__ void run(const FragT (&qf)[KS], int j_first, int stride, float c2,
                                      int G, int lane, VtTile& vt, PTile& sp) {
    const int gbase = 4 * (lane >> 4);
    for (int j0 = j_first; j0 < t_end; j0 += stride) {
      // ---- logits for the two 16-token halves
      f32x4 acc[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        acc[hh] = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) mma(acc[hh], qf[ks], kf[hh][ks]);
      }
      wave_lds_order();  // the previous block's reads of vt / sp come first
      // ---- V into LDS: bf16 rows as they are (tokens 2p, 2p+1); fp32 transposed
      {
        const int p2 = 2 * (lane & 15);
#pragma unroll
        for (int c = 0; c < NVC; ++c) {
          const int col0 = 8 * ((lane >> 4) + 4 * c);
          if constexpr (TR) {
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) store_frag(&vt[p2 + hh][col0], vf[hh][c]);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              *reinterpret_cast<float2*>(&vt[col0 + e][p2]) = make_float2(elem_f(vf[0][c], e), elem_f(vf[1][c], e));
          }
        }
      }
      if (j0 + stride < t_end) load(j0 + stride, lane);
      // ---- online softmax over the 32 tokens (rows g = gbase + i)
      float alpha[4];
      bool grew = false;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ja = j0 + (lane & 15), jb = ja + 16;
        const bool gok = gbase + i < G;
        const float xa = (ja < t_end && gok) ? acc[0][i] * c2 : -INFINITY;
        const float xb = (jb < t_end && gok) ? acc[1][i] * c2 : -INFINITY;
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
        grew |= mn != m_run[i];
        l_run[i] = l_run[i] * alpha[i] + row16_sum(pa + pb);
        m_run[i] = mn;
        if (gbase + i < GMAX) {
          sp[gbase + i][lane & 15] = from_f<T>(pa);
          sp[gbase + i][16 + (lane & 15)] = from_f<T>(pb);
        }
      }
      wave_lds_order();  // P and V are in LDS before they are read back
      // ---- O = alpha * O + P . V on MFMA (A = P rows g, B = V); alpha is exactly 1
      // where no running max grew, so the rescale is skipped when none did in the wave
      const bool rescale = __any(grew);
      const FragT pfr = ((lane & 15) < G) ? load_frag(&sp[lane & 15][8 * (lane >> 4)]) : zero_frag<T>();
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        if (rescale) {
#pragma unroll
          for (int i = 0; i < 4; ++i) oacc[nt][i] *= alpha[i];
        }
        if constexpr (TR)
          mma(oacc[nt], pfr, lds_frag_tr(&vt[0][0], LDV, 0, 16 * nt, lane));
        else
          mma(oacc[nt], pfr, load_frag(&vt[16 * nt + (lane & 15)][8 * (lane >> 4)]));
      }
    }
  }

  // o rows g < G to so[g * D + col] (a wave-private float buffer), max/sum to ml[g * 2].
  __device__ __forceinline__ void store_lds(float* so, float* ml, int G, int lane) {
    const int gbase = 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (gbase + i < G) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) so[(gbase + i) * D + 16 * nt + (lane & 15)] = oacc[nt][i];
        if ((lane & 15) == 0) {
          ml[(gbase + i) * 2 + 0] = m_run[i];
          ml[(gbase + i) * 2 + 1] = l_run[i];
        }
      }
    }
  }
};

// ---------------------------------------------------------------- correction
// CPL consecutive elements as floats (CPL = 1 or 2), one load.
template <int CPL>
__device__ __forceinline__ void load_cols(const float* p, float (&v)[CPL]) {
  if constexpr (CPL == 2) {
    const float2 t = *reinterpret_cast<const float2*>(p);
    v[0] = t.x;
    v[1] = t.y;
  } else {
    v[0] = p[0];
  }
}
template <int CPL>
__device__ __forceinline__ void load_cols(const bf16_t* p, float (&v)[CPL]) {
  if constexpr (CPL == 2) {
    const uint32_t t = *reinterpret_cast<const uint32_t*>(p);
    v[0] = __uint_as_float(t << 16);
    v[1] = __uint_as_float(t & 0xffff0000u);
  } else {
    v[0] = bf2f(p[0]);
  }
}

// Per-query inputs of the correction, lane holding columns CPL * lane ...: the query, the
// new token's key and value (the query stands in when there is none; never used) and the
// summary's key and value sums.
template <int CPL>
struct QueryCols {
  float q[CPL], kn[CPL], vn[CPL], sk[CPL], sv[CPL];
};
template <class T, int D>
__device__ __forceinline__ QueryCols<D / 64> load_query_cols(const DecodeArgs& a, int bh, int g,
                                                             int lane) {
  constexpr int CPL = D / 64;
  const int col = lane * CPL;
  const T* q = reinterpret_cast<const T*>(a.q) + ((size_t)bh * a.G + g) * D + col;
  const bool has_new = a.k_new != nullptr;
  QueryCols<CPL> r;
  load_cols<CPL>(q, r.q);
  load_cols<CPL>(has_new ? reinterpret_cast<const T*>(a.k_new) + (size_t)bh * D + col : q, r.kn);
  load_cols<CPL>(has_new ? reinterpret_cast<const T*>(a.v_new) + (size_t)bh * D + col : q, r.vn);
  load_cols<CPL>(a.s_k + (size_t)bh * D + col, r.sk);
  load_cols<CPL>(a.s_v + (size_t)bh * D + col, r.sv);
  return r;
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

// One query head (one wave): fold the new token into the merged cache state (M, l, o),
// mix in f_E_hat = v_bar + scale / n_e * S_tilde q (sqv, used when use_sq) with the
// Jensen weight, write out / lse / w_R.
template <class T, int D>
__device__ __forceinline__ void finish_query(const DecodeArgs& a, int bh, int g, int lane,
                                             float M, float l, float (&o)[D / 64],
                                             const QueryCols<D / 64>& qc, const float (&sqv)[D / 64],
                                             bool use_sq, int ne, bool add_new) {
  constexpr int CPL = D / 64;
  if (a.order < 0) ne = 0;  // no correction: the output is f_R, as with an empty summary
  float dot_k = 0.f, dot_s = 0.f;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    dot_k += qc.q[c] * qc.kn[c];
    dot_s += qc.q[c] * qc.sk[c];
  }
  dot_k = wave_sum(dot_k);
  dot_s = wave_sum(dot_s);
  if (add_new) {  // the new token, after the cache rows (logit in log2 units)
    const float x = dot_k * a.scale * kLog2e;
    const float mn = fmaxf(M, x);
    const float r = fast_exp2(M - mn), w = fast_exp2(x - mn);
    l = l * r + w;
#pragma unroll
    for (int c = 0; c < CPL; ++c) o[c] = o[c] * r + w * qc.vn[c];
    M = mn;
  }
  const Mix mx = mix_weights(M, l, ne, dot_s, a.scale);
  const float inv_n = ne > 0 ? 1.f / (float)ne : 0.f;
  const int pair = bh * a.G + g;
  T* out = reinterpret_cast<T*>(a.out) + (size_t)pair * D + lane * CPL;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const float f_r = (l > 0.f) ? o[c] / l : 0.f;
    float res = f_r;
    if (ne > 0) {
      float fe = qc.sv[c] * inv_n;
      if (use_sq) fe += a.scale * inv_n * sqv[c];
      res = mx.w_r * f_r + (1.f - mx.w_r) * fe;
    }
    out[c] = from_f<T>(res);
  }
  if (lane == 0) {
    if (a.lse_out) a.lse_out[pair] = mx.log_zr;
    if (a.w_r_out) a.w_r_out[pair] = mx.w_r;
  }
}

// ---------------------------------------------------------------- fused launch
template <class T, int D, int GMAX, int PREP>
__global__ void __launch_bounds__(256) k_decode_fused(DecodeArgs a) {
  typedef BlockAttn<T, D, GMAX> BA;
  constexpr int CPL = D / 64;
  constexpr int KS = D / 32;
  // per-wave V tile; after the wave's blocks it holds the wave's o rows as floats
  constexpr int VT_BYTES = (int)sizeof(typename BA::VtTile);
  static_assert(VT_BYTES >= GMAX * D * 4, "o rows fit in the V tile");
  __shared__ __align__(16) unsigned char s_vt[4][VT_BYTES];
  __shared__ __align__(16) T s_p[4][16][BA::TB + BA::PT];
  __shared__ float s_ml[4][GMAX * 2];
  __shared__ float s_sq[GMAX * D];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int head = blockIdx.x;
  const int G = a.G;
  const T* qh = reinterpret_cast<const T*>(a.q) + (size_t)head * G * D;
  typename BA::VtTile& vt = *reinterpret_cast<typename BA::VtTile*>(s_vt[wave]);

  typename BA::FragT qf[KS];
  load_query_frags<T, D>(qh, G, lane, qf);
  const bool sq_rows = a.nsq > 0 && 32 * wave < D;
  SqRows<T, D, PREP> sq;
  if (sq_rows) sq.load(a, head, 32 * wave, lane);
  const QueryCols<CPL> qc = load_query_cols<T, D>(a, head, min(wave, G - 1), lane);
  const int ne = a.n_e[head];

  BA ba;
  ba.kc = reinterpret_cast<const T*>(a.k_cache) + (size_t)head * a.cap * D;
  ba.vc = reinterpret_cast<const T*>(a.v_cache) + (size_t)head * a.cap * D;
  ba.init();
  // The wave's first block is requested together with lens, bounded by the capacity only
  // (rows 32w.. exist whatever lens is); once lens is known, V rows at or past it are
  // cleared (they may hold any bits) and their logits are masked like any row past t_end.
  ba.t_end = a.cap;
  ba.load(BA::TB * wave, lane);
  const HeadLen hl = head_len(a, a.lens[head]);
  ba.t_end = hl.cache_len;
  if (BA::TB * (wave + 1) > ba.t_end) ba.clear_v_past_end(BA::TB * wave, lane);
  if (wave == 0 && lane == 0 && a.k_new != nullptr && !hl.can_append) atomicOr(a.flag, 1);
  if (sq_rows) sq.compute(a, qf, 32 * wave, lane, s_sq);
  ba.run(qf, BA::TB * wave, 4 * BA::TB, a.scale * kLog2e, G, lane, vt, s_p[wave]);
  wave_lds_order();  // the last block's reads of the V tile come before it is reused
  ba.store_lds(reinterpret_cast<float*>(s_vt[wave]), s_ml[wave], G, lane);
  // the copy of the new token into the cache: nothing here reads that row (the token is
  // attended to from k_new / v_new), so it waits until the wave's own rows are used
  if (wave == 3 && hl.can_append) append_row<T, D>(a, head, hl.old_len, lane);
  __syncthreads();

  // one wave per query: merge the four waves' states, then the new token and correction
  for (int g = wave; g < G; g += 4) {
    const QueryCols<CPL> qg = g == wave ? qc : load_query_cols<T, D>(a, head, g, lane);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_ml[w][2 * g]);
    float l = 0.f, o[CPL], sqv[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      o[c] = 0.f;
      sqv[c] = s_sq[g * D + lane * CPL + c];
    }
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float wt = fast_exp2(s_ml[w][2 * g] - M);
        l += s_ml[w][2 * g + 1] * wt;
        const float* so = reinterpret_cast<const float*>(s_vt[w]) + g * D + lane * CPL;
#pragma unroll
        for (int c = 0; c < CPL; ++c) o[c] += so[c] * wt;
      }
    }
    finish_query<T, D>(a, head, g, lane, M, l, o, qg, sqv, a.nsq > 0, ne, hl.can_append);
  }
  if (threadIdx.x == 0 && hl.can_append) a.lens[head] = hl.old_len + 1;
}

// ---------------------------------------------------------------- split launch
// CPL consecutive elements of a row as floats (16 or 32 bytes, one or two loads), and the
// converse store.
template <int CPL>
__device__ __forceinline__ void load_span(const float* p, float (&v)[CPL]) {
#pragma unroll
  for (int c = 0; c < CPL; c += 4) {
    const float4 t = *reinterpret_cast<const float4*>(p + c);
    v[c] = t.x; v[c + 1] = t.y; v[c + 2] = t.z; v[c + 3] = t.w;
  }
}
template <int CPL>
__device__ __forceinline__ void load_span(const bf16_t* p, float (&v)[CPL]) {
  static_assert(CPL == 4 || CPL == 8, "4 or 8 columns");
  uint32_t w[CPL / 2];
  if constexpr (CPL == 8) {
    const uint4 t = *reinterpret_cast<const uint4*>(p);
    w[0] = t.x; w[1] = t.y; w[2] = t.z; w[3] = t.w;
  } else {
    const uint2 t = *reinterpret_cast<const uint2*>(p);
    w[0] = t.x; w[1] = t.y;
  }
#pragma unroll
  for (int c = 0; c < CPL / 2; ++c) {
    v[2 * c] = __uint_as_float(w[c] << 16);
    v[2 * c + 1] = __uint_as_float(w[c] & 0xffff0000u);
  }
}
template <int CPL>
__device__ __forceinline__ void store_span(float* p, const float (&v)[CPL]) {
#pragma unroll
  for (int c = 0; c < CPL; c += 4)
    *reinterpret_cast<float4*>(p + c) = make_float4(v[c], v[c + 1], v[c + 2], v[c + 3]);
}
template <int CPL>
__device__ __forceinline__ void store_span(bf16_t* p, const float (&v)[CPL]) {
  uint32_t w[CPL / 2];
#pragma unroll
  for (int c = 0; c < CPL / 2; ++c) w[c] = (uint32_t)f2bf(v[2 * c]) | ((uint32_t)f2bf(v[2 * c + 1]) << 16);
  if constexpr (CPL == 8) *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  else *reinterpret_cast<uint2*>(p) = make_uint2(w[0], w[1]);
}

// Merge of one KV head by the last wave of the split launch to count itself in: four
// query heads at a time, query g0 + lane / 16 in each 16-lane row, the lane holding columns
// CPL * (lane % 16) ... + CPL.  The slices' (max, sum) pairs are combined in slice order,
// sixteen at a time (lane % 16 = slice), their o rows SUBR at a time; then the new token is
// folded in and the moment correction applied, as in the single-launch path.  The slices'
// partials and the S_tilde q rows are read with agent-scope loads.
template <class T, int D>
__device__ __forceinline__ void merge_head(const DecodeArgs& a, int head, int lane) {
  constexpr int CPL = D / 16;  // columns per lane
  constexpr int SUBR = 4;      // slices whose o rows are in flight together
  const int r = lane & 15, c0 = CPL * r, G = a.G;
  const HeadLen hl = head_len(a, a.lens[head]);
  const int ne = a.order < 0 ? 0 : a.n_e[head];  // order -1: the output is f_R
  const int n_live = live_slices(a, hl.cache_len);
  const int last = max(n_live, 1) - 1;
  const bool use_sq = a.nsq > 0;
  for (int g0 = 0; g0 < G; g0 += 4) {
    const bool gok = g0 + (lane >> 4) < G;
    const int g = min(g0 + (lane >> 4), G - 1);  // rows past G repeat the last query, unstored
    const size_t pair = (size_t)head * G + g;
    auto ml_of = [&](int s) {
      return ld_agent2(a.part_ml + (((size_t)head * a.nsplit + min(s, last)) * G + g) * 2);
    };
    auto o_row = [&](int s, float (&v)[CPL]) {
      const float* p = a.part_o + (((size_t)head * a.nsplit + min(s, last)) * G + g) * D + c0;
#pragma unroll
      for (int c = 0; c < CPL; c += 2) {
        const float2 t = ld_agent2(p + c);
        v[c] = t.x;
        v[c + 1] = t.y;
      }
    };
    // every read of the query's inputs before the first reduction
    float2 ml = ml_of(r);
    float ov[SUBR][CPL];
#pragma unroll
    for (int u = 0; u < SUBR; ++u) o_row(u, ov[u]);
    float sqv[CPL], q[CPL], kn[CPL], vn[CPL], sk[CPL], sv[CPL];
    if (use_sq) {
      const float* p = a.sq + pair * D + c0;
#pragma unroll
      for (int c = 0; c < CPL; c += 2) {
        const float2 t = ld_agent2(p + c);
        sqv[c] = t.x;
        sqv[c + 1] = t.y;
      }
    }
    const T* qp = reinterpret_cast<const T*>(a.q) + pair * D + c0;
    const bool has_new = a.k_new != nullptr;
    load_span<CPL>(qp, q);
    load_span<CPL>(has_new ? reinterpret_cast<const T*>(a.k_new) + (size_t)head * D + c0 : qp, kn);
    load_span<CPL>(has_new ? reinterpret_cast<const T*>(a.v_new) + (size_t)head * D + c0 : qp, vn);
    load_span<CPL>(a.s_k + (size_t)head * D + c0, sk);
    load_span<CPL>(a.s_v + (size_t)head * D + c0, sv);

    float M = -INFINITY, l = 0.f, o[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) o[c] = 0.f;
    for (int s0 = 0; s0 < n_live; s0 += 16) {
      if (s0 > 0) ml = ml_of(s0 + r);
      const bool live = s0 + r < n_live;
      const float mn = fmaxf(M, row16_max(live ? ml.x : -INFINITY));
      if (mn == -INFINITY) continue;  // nothing attended to so far (uniform over the row)
      const float rs = fast_exp2(M - mn);
      const float w = live ? fast_exp2(ml.x - mn) : 0.f;
      l = l * rs + row16_sum(live ? ml.y * w : 0.f);
#pragma unroll
      for (int c = 0; c < CPL; ++c) o[c] *= rs;
      M = mn;
      const int cn = min(16, n_live - s0);
      for (int u0 = 0; u0 < cn; u0 += SUBR) {
        if (s0 + u0 > 0) {
#pragma unroll
          for (int u = 0; u < SUBR; ++u) o_row(s0 + u0 + u, ov[u]);
        }
#pragma unroll
        for (int u = 0; u < SUBR; ++u) {
          const float wu = __shfl(w, (lane & 48) + min(u0 + u, 15));
          if (u0 + u < cn) {
#pragma unroll
            for (int c = 0; c < CPL; ++c) o[c] += wu * ov[u][c];
          }
        }
      }
    }
    // the new token after the cache rows, then the correction (finish_query's arithmetic
    // with the dot products summed over the row's 16 lanes)
    float dot_k = 0.f, dot_s = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      dot_k += q[c] * kn[c];
      dot_s += q[c] * sk[c];
    }
    dot_k = row16_sum(dot_k);
    dot_s = row16_sum(dot_s);
    if (hl.can_append) {
      const float x = dot_k * a.scale * kLog2e;
      const float mn = fmaxf(M, x);
      const float rr = fast_exp2(M - mn), w = fast_exp2(x - mn);
      l = l * rr + w;
#pragma unroll
      for (int c = 0; c < CPL; ++c) o[c] = o[c] * rr + w * vn[c];
      M = mn;
    }
    const Mix mx = mix_weights(M, l, ne, dot_s, a.scale);
    const float inv_n = ne > 0 ? 1.f / (float)ne : 0.f;
    float res[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const float f_r = (l > 0.f) ? o[c] / l : 0.f;
      res[c] = f_r;
      if (ne > 0) {
        float fe = sv[c] * inv_n;
        if (use_sq) fe += a.scale * inv_n * sqv[c];
        res[c] = mx.w_r * f_r + (1.f - mx.w_r) * fe;
      }
    }
    if (gok) {
      store_span<CPL>(reinterpret_cast<T*>(a.out) + pair * D + c0, res);
      if (r == 0) {
        if (a.lse_out) a.lse_out[pair] = mx.log_zr;
        if (a.w_r_out) a.w_r_out[pair] = mx.w_r;
      }
    }
  }
  if (lane == 0) {
    // every other wave of the head has counted itself in, and so has read lens
    __hip_atomic_store(a.cnt + head, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (hl.can_append) a.lens[head] = hl.old_len + 1;
  }
}

// One launch, a 1-D grid of single-wave workgroups: n_heads x nsq waves of 32 rows of
// S_tilde q, then n_heads x nsplit token slices.  Each wave writes its result (S_tilde q
// rows, or the slice's unnormalised (o, max, sum)), then counts itself in on its head's
// counter; the wave that completes the count merges the head (merge_head) and sets the
// counter back to zero for the next call.
// bf16: three waves per SIMD fit without spills (the accumulators move from AGPRs to
// VGPRs); the fp32 form keeps the compiler's choice.
template <class T, int D, int GMAX, int PREP>
__global__ void __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(sizeof(T) == 2 ? 3 : 1)))
k_decode_slice(DecodeArgs a) {
  typedef BlockAttn<T, D, GMAX> BA;
  constexpr int KS = D / 32;
  constexpr int VT_BYTES = (int)sizeof(typename BA::VtTile);
  static_assert(VT_BYTES >= GMAX * D * 4, "o rows fit in the V tile");
  __shared__ __align__(16) unsigned char s_vt[VT_BYTES];
  __shared__ __align__(16) T s_p[16][BA::TB + BA::PT];
  __shared__ float s_ml[GMAX * 2];

  // Workgroups reach the XCDs round-robin by id, so each kind of wave is numbered
  // contiguously: the S_tilde q waves first (head-major), then the token slices
  // (head-major); either kind then spreads evenly over the XCDs whatever nsq and nsplit.
  const int lane = threadIdx.x;
  const int n_sq = a.n_heads * a.nsq;
  const bool is_sq = (int)blockIdx.x < n_sq;
  const int idx = is_sq ? (int)blockIdx.x : (int)blockIdx.x - n_sq;
  const int nsq = max(a.nsq, 1);  // no S_tilde q waves when a.nsq = 0 (is_sq is false)
  const int head = is_sq ? idx / nsq : idx / a.nsplit;   // b * Hkv + h
  const int G = a.G;
  const T* qh = reinterpret_cast<const T*>(a.q) + (size_t)head * G * D;
  // the query fragments are requested after the wave's other reads: zeroing the rows past
  // G right after the reads would otherwise hold those back until the queries arrive
  typename BA::FragT qf[KS];
  if (is_sq) {
    const int r0 = 32 * (idx % nsq);
    SqRows<T, D, PREP> sq;
    sq.load(a, head, r0, lane);
    load_query_frags<T, D>(qh, G, lane, qf);
    sq.template compute<true>(a, qf, r0, lane, a.sq + (size_t)head * G * D);
  } else {
    const int split = idx % a.nsplit;
    const HeadLen hl = head_len(a, a.lens[head]);
    const int t0 = split * a.split_len;
    BA ba;
    ba.kc = reinterpret_cast<const T*>(a.k_cache) + (size_t)head * a.cap * D;
    ba.vc = reinterpret_cast<const T*>(a.v_cache) + (size_t)head * a.cap * D;
    ba.t_end = max(t0, min(t0 + a.split_len, hl.cache_len));
    ba.init();
    ba.load(t0, lane);  // rows clamped into the cache for an empty slice; never used
    load_query_frags<T, D>(qh, G, lane, qf);
    if (a.k_new != nullptr && !hl.can_append && split == 0 && lane == 0) atomicOr(a.flag, 1);
    // the slice whose range holds row old_len (the last slice for rows past the split)
    if (hl.can_append && min(hl.old_len / a.split_len, a.nsplit - 1) == split)
      append_row<T, D>(a, head, hl.old_len, lane);
    if (t0 < ba.t_end) {  // an empty slice writes nothing: the merge skips it
      typename BA::VtTile& vt = *reinterpret_cast<typename BA::VtTile*>(s_vt);
      ba.run(qf, t0, BA::TB, a.scale * kLog2e, G, lane, vt, s_p);
      // partials through LDS so that each lane stores whole 8-byte pairs
      wave_lds_order();
      float* so = reinterpret_cast<float*>(s_vt);
      ba.store_lds(so, s_ml, G, lane);
      wave_lds_order();
      const size_t pbase = ((size_t)head * a.nsplit + split) * G;
      float* po = a.part_o + pbase * D;
      for (int c = lane; c < G * D / 2; c += kWave) st_agent2(po + 2 * c, so[2 * c], so[2 * c + 1]);
      if (lane < G) st_agent2(a.part_ml + (pbase + lane) * 2, s_ml[2 * lane], s_ml[2 * lane + 1]);
    }
  }
  // count in; the wave completing the head's count merges it
  stores_complete();
  int prior = 0;
  if (lane == 0) prior = atomicAdd(a.cnt + head, 1);
  prior = __builtin_amdgcn_readfirstlane(prior);
  if (prior != a.nsq + a.nsplit - 1) return;
  loads_after_count();
  merge_head<T, D>(a, head, lane);
}

template <class T, int D, int GMAX, int PREP>
static hipError_t launch_decode_p(const DecodeArgs& a, hipStream_t st) {
  if (a.fused) {
    hipLaunchKernelGGL((k_decode_fused<T, D, GMAX, PREP>), dim3(a.n_heads), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  const unsigned grid = (unsigned)a.n_heads * (unsigned)(a.nsq + a.nsplit);
  hipLaunchKernelGGL((k_decode_slice<T, D, GMAX, PREP>), dim3(grid), dim3(64), 0, st, a);
  return hipGetLastError();
}

template <class T, int D, int GMAX>
static hipError_t launch_decode_t(const DecodeArgs& a, hipStream_t st) {
  if (a.summary == 1) return launch_decode_p<T, D, GMAX, 1>(a, st);
  if (a.summary == 3) return launch_decode_p<T, D, GMAX, 3>(a, st);
  if constexpr (sizeof(T) == 2) {
    if (a.summary == 2) return launch_decode_p<T, D, GMAX, 2>(a, st);
  }
  return launch_decode_p<T, D, GMAX, 0>(a, st);
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

template <class T, int D>
static hipError_t launch_prepare_t(const DecodeArgs& a, void* prepared, hipStream_t st) {
  hipLaunchKernelGGL((k_prepare_summary<T, D>), dim3((D * D / 8 + 255) / 256, a.n_heads), dim3(256), 0,
                     st, a, prepared, a.summary == 2 ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_prepare_summary(const DecodeArgs& a, void* prepared, bool bf16, int d, hipStream_t st) {
  if (bf16) return d == 64 ? launch_prepare_t<bf16_t, 64>(a, prepared, st) : launch_prepare_t<bf16_t, 128>(a, prepared, st);
  return d == 64 ? launch_prepare_t<float, 64>(a, prepared, st) : launch_prepare_t<float, 128>(a, prepared, st);
}

}  // namespace mkv
