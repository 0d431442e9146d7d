// Decode step with moment-informed eviction: Algorithm 1 Phase 1 (one eviction), then the
// corrected attention of Phase 2 over the new cache and summary, reading the cache once.
//
// k_evict_attn: about one NW-wave workgroup per CU (the LDS holds S_tilde and a V tile
//   per wave), each taking an equal share of the flattened (head, 32-row block) range.
//   For each head its share touches, the workgroup forms the summary's clamped covariance
//   S_tilde = S - s_v s_k^T / n_e (entries below tau set to zero; zero when n_e = 0) from
//   the raw moments into LDS (hi / lo bf16 planes for bf16 caches, fp32 otherwise) if the
//   head evicts this call, while each wave's first block is in flight.  Each wave then
//   takes the blocks w, w + NW, ... of the share, the new token included (row lens, read
//   from k_new / v_new); lane l holds rows j0 + 2 (l % 16) + {0, 1} at dims
//   32 c + 8 (l / 16) + e.  Per block:
//     x_gj = scale log2(e) q_g . k_j on MFMA (base-2 logits of the G queries);
//     if the head evicts, the records x_gj and y_j = log2 ||r_j||, with
//       r_j = v_j - v_bar - (scale / n_e) S_tilde k_j (Eq. residual); S_tilde k_j runs on
//       MFMA (S_tilde rows from LDS as A, the K fragments of the logits as B), its A rows
//       ordered so that each lane receives the dims of v_j it holds, so r_j and its
//       squared norm are formed in registers;
//     the attention over every row (which one leaves is not known yet): online softmax
//       in the base-2 domain and P.V on MFMA, V read back out of LDS with the transposing
//       LDS read (bf16) or written transposed (fp32).  The running
//       max after the block is recorded, so that a row's term can later be taken out
//       exactly as it was accumulated.
//   The waves' states are merged in LDS and written as one partial state of the head.
// k_evict_finish: one workgroup per head combines the head's partial states in order,
//   then selects and finishes:
//   log2 Z_g over R from the logits, the group-mean softmax weight
//   alpha_j = mean_g 2^(x_gj - log2 Z_g) in the log domain (no weight underflows), the
//   argmin of log2 alpha_j + y_j (the lowest row on ties), the rank-one update n_e += 1,
//   s_k += k*, s_v += v*, S += v* k*^T (App. A.1 Eq. app_update) and the move of the last
//   row into the freed slot.  The evicted row's term leaves the attention state; where it
//   held nearly all of a query's mass (the rest would then keep few significant digits)
//   the attention over the new cache is computed again instead.  Last, S_tilde q from the
//   updated summary and the correction w_R f_R + (1 - w_R) (v_bar + (scale / n_e)
//   S_tilde q) with the Jensen estimate of the evicted mass (Eqs. fhat, jensen, fused).
// Short caches: k_evict_attn without the attention, one workgroup per head (two per CU),
//   scores the head's rows as above, then selects and finishes as k_evict_finish does,
//   with the attention over the new cache computed after the update (rows it has just
//   read, mostly from L2; V tiles in the LDS that held S_tilde).
#include <climits>

#include "mkv_bf16.h"
#include "mkv_device.h"
#include "mkv_evict.h"

namespace mkv {

namespace {

constexpr int kEvTB = 32;           // rows per block
constexpr int kFinWaves = 4;        // waves of a finishing workgroup
constexpr int kMaxSlices = 64;      // partial states merged by one finishing wave
constexpr float kRedoRatio = 16.f;  // recompute when a removed term exceeds this many
                                    // times what remains of a query's sum

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Orders the wave's own LDS writes and reads for the compiler.  A wave's LDS operations
// are carried out in issue order, so lanes of one wave exchanging data through LDS need
// no hardware wait beyond that.
__device__ __forceinline__ void wave_lds_order() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// The thread's index as a value the compiler cannot move: per-thread offsets derived from
// it are formed where a segment needs them instead of being hoisted out of the loop over
// segments (where, kept live across the block loop, they would be spilled).
__device__ __forceinline__ int tid_here() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

// x * y rounded on its own, never fused into a following add: the scaled logits are
// stored and used again later, and must be the same bits in both places.
__device__ __forceinline__ float mul_nofuse(float x, float y) {
#pragma clang fp contract(off)
  return x * y;
}

// S_tilde in LDS.
template <class T, int D> struct SumLds;
template <int D> struct SumLds<bf16_t, D> {
  bf16_t hi[D * D];
  bf16_t lo[D * D];
  // Element (row, col).  Rows are unpadded; the 16-byte chunks of a row are XOR-swizzled
  // so that the 16 rows one MFMA operand read touches (r + {0..3, 8..11, 16..19, 24..27})
  // sit in 16 different chunks, i.e. in different banks (8 chunks for D = 64).
  static __device__ __forceinline__ int at(int row, int col) {
    constexpr int NC = D / 8;
    const int f = ((row & 3) | (((row >> 3) & 3) << 2)) & (NC - 1);
    return row * D + (((col >> 3) ^ f) << 3) + (col & 7);
  }
};
template <int D> struct SumLds<float, D> {
  static constexpr int RS = D + 4;
  float st[D * RS];
  static __device__ __forceinline__ int at(int row, int col) { return row * RS + col; }
};

__device__ __forceinline__ bf16x8 lds_frag(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}
__device__ __forceinline__ f32x8 lds_frag(const float* p) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  f32x8 r;
  r[0] = a.x; r[1] = a.y; r[2] = a.z; r[3] = a.w;
  r[4] = b.x; r[5] = b.y; r[6] = b.z; r[7] = b.w;
  return r;
}

// S_tilde of one head into LDS; every thread handles D*D/8/NT chunks of 8 entries of a
// row.  n_e is read after the rows of S and everything that depends on it follows a
// scheduling barrier, so that no read here waits behind the caller's reads in flight
// (the compiler moves a uniform value read from memory to a scalar register at once).
// Returns n_e.
template <class T, int D, int NT>
__device__ __forceinline__ int build_summary(const EvictArgs& e, int head, SumLds<T, D>& sm) {
  constexpr int PER = D * D / 8 / NT;
  static_assert(PER >= 1 && (D * D / 8) % NT == 0, "whole chunks per thread");
  const int tid = tid_here();
  const int c0 = 8 * (tid % (D / 8));
  const float* Sh = e.S + (size_t)head * D * D;
  const f32x8 skc = load_frag(e.s_k + (size_t)head * D + c0);
  f32x8 raw[PER];
  float sv[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int row = (tid + NT * u) / (D / 8);
    raw[u] = load_frag(Sh + (size_t)row * D + c0);
    sv[u] = e.s_v[(size_t)head * D + row];
  }
  const int ne = e.n_e[head];
  __builtin_amdgcn_sched_barrier(0);
  const float inv_n = 1.f / (float)max(ne, 1);  // unused when ne <= 0 (S_tilde = 0)
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int row = (tid + NT * u) / (D / 8);
    float st[8];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      const float t = raw[u][x] - sv[u] * (skc[x] * inv_n);
      st[x] = (ne <= 0 || fabsf(t) < e.tau) ? 0.f : t;
    }
    if constexpr (sizeof(T) == 2) {
      uint32_t h[4], l[4];
#pragma unroll
      for (int x = 0; x < 8; x += 2) bf16_split_pair(st[x], st[x + 1], h[x / 2], l[x / 2]);
      const int at = SumLds<T, D>::at(row, c0);
      *reinterpret_cast<uint4*>(&sm.hi[at]) = make_uint4(h[0], h[1], h[2], h[3]);
      *reinterpret_cast<uint4*>(&sm.lo[at]) = make_uint4(l[0], l[1], l[2], l[3]);
    } else {
      float4* P = reinterpret_cast<float4*>(&sm.st[SumLds<T, D>::at(row, c0)]);
      P[0] = make_float4(st[0], st[1], st[2], st[3]);
      P[1] = make_float4(st[4], st[5], st[6], st[7]);
    }
  }
  return ne;
}

// The new token: the wave given the job copies k_new / v_new to cache row `row`, 16 bytes
// per lane; the read and the write may also be issued apart (append_read, append_write).
template <class T, int D>
__device__ __forceinline__ uint4 append_read(const EvictArgs& e, int head, int lane) {
  constexpr int NV = D * (int)sizeof(T) / 16;
  const bool is_v = lane >= NV;
  const uint4* src = reinterpret_cast<const uint4*>(
      reinterpret_cast<const T*>(is_v ? e.v_new : e.k_new) + (size_t)head * D) + lane % NV;
  return *src;  // every lane reads inside the row; lanes past 2 NV write nothing
}
template <class T, int D>
__device__ __forceinline__ void append_write(const EvictArgs& e, int head, int row, int lane,
                                             const uint4& piece) {
  constexpr int NV = D * (int)sizeof(T) / 16;
  if (lane < 2 * NV) {
    T* cache = reinterpret_cast<T*>(lane >= NV ? e.v_cache : e.k_cache);
    reinterpret_cast<uint4*>(cache + ((size_t)head * e.cap + row) * D)[lane % NV] = piece;
  }
}
template <class T, int D>
__device__ __forceinline__ void append_new_row(const EvictArgs& e, int head, int row, int lane) {
  append_write<T, D>(e, head, row, lane, append_read<T, D>(e, head, lane));
}

// Whether this call evicts from the head: the new row fits in the cache and in the
// row bound, and the cache then holds more than `budget` rows.
__device__ __forceinline__ bool head_evicts(const EvictArgs& e, int old_len) {
  return old_len >= 0 && old_len < e.cap && old_len + 1 <= e.max_len && old_len + 1 > e.budget;
}

// The G query rows of a head into LDS (rows past G, up to 16, zero): the A operand of
// the logits.  load() issues the reads, store() writes them once other work is out.
template <class T, int D, int NT>
struct QueryRows {
  static constexpr int QRS = D + 16 / (int)sizeof(T);  // rows padded by 16 bytes
  static constexpr int QPR = D * (int)sizeof(T) / 16;  // 16-byte pieces per row
  static constexpr int QPT = (16 * QPR + NT - 1) / NT;
  uint4 qv[QPT];
  __device__ __forceinline__ void load(const EvictArgs& e, int head) {
    const T* qh = reinterpret_cast<const T*>(e.q) + (size_t)head * e.G * D;
    const int tid = tid_here();
#pragma unroll
    for (int u = 0; u < QPT; ++u) {
      const int p = tid + NT * u, row = p / QPR;
      qv[u] = (p < 16 * QPR && row < e.G)
                  ? *reinterpret_cast<const uint4*>(qh + (size_t)row * D + (p % QPR) * (16 / (int)sizeof(T)))
                  : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(T* s_q) const {
    const int tid = tid_here();
#pragma unroll
    for (int u = 0; u < QPT; ++u) {
      const int p = tid + NT * u;
      if (p < 16 * QPR)
        *reinterpret_cast<uint4*>(&s_q[(p / QPR) * QRS + (p % QPR) * (16 / (int)sizeof(T))]) = qv[u];
    }
  }
};

// ---------------------------------------------------------------- attention of a wave
// Online-softmax attention state of one wave over its blocks; query g = 4 (l / 16) + i
// sits in MFMA row g, lane l holding entry i.
template <class T, int D, int GM>
struct EvAttn {
  static constexpr int KS = D / 32;
  static constexpr int NOT = D / 16;              // 16-column output tiles of P.V
  static constexpr int PT = 16 / (int)sizeof(T);  // LDS row padding (16 bytes)
  static constexpr int QRS = D + 16 / (int)sizeof(T);
  static constexpr bool TR = sizeof(T) == 2;       // bf16: V kept in its own layout
  static constexpr int LDV = D + 16;               // bf16 V rows padded by 32 bytes
  typedef typename Frag<T>::type FragT;
  // bf16: the block's V rows as they are, read back transposed as MFMA operands; fp32:
  // V^T, written transposed
  typedef typename Pick<TR, T[kEvTB][LDV], T[D][kEvTB + PT]>::type VtTile;
  typedef T PTile[GM][kEvTB + PT];
  static_assert(sizeof(VtTile) >= GM * D * sizeof(float), "o rows fit in the V tile");

  float m_run[4], l_run[4];
  f32x4 oacc[NOT];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < 4; ++i) { m_run[i] = -INFINITY; l_run[i] = 0.f; }
#pragma unroll
    for (int nt = 0; nt < NOT; ++nt) oacc[nt] = zero4();
  }

  // Base-2 logits c2 q_g . k of the rows j0 + 2 (l % 16) + hh in x[hh] (queries from LDS).
  static __device__ __forceinline__ void logits(const T* s_q, const FragT (&kf)[2][KS], float c2,
                                                int lane, f32x4 (&x)[2]) {
    const int r16 = lane & 15, q4 = lane >> 4;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      f32x4 acc = zero4();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) mma(acc, lds_frag(&s_q[r16 * QRS + 32 * ks + 8 * q4]), kf[hh][ks]);
#pragma unroll
      for (int i = 0; i < 4; ++i) x[hh][i] = mul_nofuse(acc[i], c2);
    }
  }

  // One block at j0: x the base-2 logits (rows at or past t_end masked), vf the V
  // fragments of the same rows (dims 32 c + 8 (l / 16) + e).
  __device__ __forceinline__ void block(const f32x4 (&x)[2], const FragT (&vf)[2][KS], int j0,
                                        int t_end, int G, int lane, VtTile& vt, PTile& sp) {
    const int r16 = lane & 15, q4 = lane >> 4, p2 = 2 * r16;
    wave_lds_order();  // the previous block's reads of vt / sp come first
    // V into LDS: bf16 rows as they are (the lane's rows p2, p2 + 1); fp32 transposed, one
    // 64-bit word per dim holding the lane's two rows
#pragma unroll
    for (int c = 0; c < KS; ++c) {
      const int col0 = 32 * c + 8 * q4;
      if constexpr (TR) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) store_frag(&vt[p2 + hh][col0], vf[hh][c]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          *reinterpret_cast<float2*>(&vt[col0 + e][p2]) = make_float2(elem_f(vf[0][c], e), elem_f(vf[1][c], e));
      }
    }
    // online softmax over the 32 rows
    float alpha[4];
    bool grew = false;
    const int ja = j0 + p2;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = 4 * q4 + i;
      const bool gok = g < G;
      const float xa = (ja < t_end && gok) ? x[0][i] : -INFINITY;
      const float xb = (ja + 1 < t_end && gok) ? x[1][i] : -INFINITY;
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
      if (g < GM) {
        if constexpr (sizeof(T) == 2) {
          *reinterpret_cast<uint32_t*>(&sp[g][p2]) = bf16_pair(pa, pb);
        } else {
          sp[g][p2] = pa;
          sp[g][p2 + 1] = pb;
        }
      }
    }
    wave_lds_order();  // P and V are in LDS before they are read back
    // O = alpha O + P . V (A = P rows g, B = V); alpha is exactly 1 where no running
    // max grew, so the rescale is skipped when none did in the whole wave
    const bool rescale = __any(grew);
    const FragT pfr = (r16 < G) ? load_frag(&sp[min(r16, GM - 1)][8 * q4]) : zero_frag<T>();
#pragma unroll
    for (int nt = 0; nt < NOT; ++nt) {
      if (rescale) {
#pragma unroll
        for (int i = 0; i < 4; ++i) oacc[nt][i] *= alpha[i];
      }
      if constexpr (TR)
        mma(oacc[nt], pfr, lds_frag_tr(&vt[0][0], LDV, 0, 16 * nt, lane));
      else
        mma(oacc[nt], pfr, load_frag(&vt[16 * nt + r16][8 * q4]));
    }
  }

  // A weight as the P tile holds it (rounded to the element type).
  static __device__ __forceinline__ float p_held(float p) {
    if constexpr (sizeof(T) == 2) return __uint_as_float(bf16_pair(p, 0.f) << 16);
    else return p;
  }

  // Running max of query 4 (l / 16) + (l % 4) (the same in the 16 lanes of a row).
  __device__ __forceinline__ float m_of_lane(int lane) const {
    const int i = lane & 3;
    return i == 0 ? m_run[0] : (i == 1 ? m_run[1] : (i == 2 ? m_run[2] : m_run[3]));
  }

  // o rows g < G to so[g * D + col], (max, sum) to ml[2 g].
  __device__ __forceinline__ void store_lds(float* so, float* ml, int G, int lane) const {
    const int r16 = lane & 15, q4 = lane >> 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = 4 * q4 + i;
      if (g < G) {
#pragma unroll
        for (int nt = 0; nt < NOT; ++nt) so[g * D + 16 * nt + r16] = oacc[nt][i];
        if (r16 == 0) {
          ml[2 * g] = m_run[i];
          ml[2 * g + 1] = l_run[i];
        }
      }
    }
  }
};

// Merged attention state of the queries g = wave + NW k a wave handles (lane l holds
// columns CPL l ...).
template <int GM, int NW, int D>
struct QState {
  static constexpr int KQ = (GM + NW - 1) / NW;
  static constexpr int CPL = D / 64;
  float M[KQ], l[KQ], o[KQ][CPL];
};

// Merge of nw wave states (wave w's o rows as floats at so + w * stride, its (max, sum)
// at ml[w * 2 GM + 2 g]) in wave order.
template <int GM, int NW, int D>
__device__ __forceinline__ void merge_waves(QState<GM, NW, D>& qs, const float* so, int stride,
                                            const float* ml, int nw, int G, int wave, int lane) {
  constexpr int CPL = D / 64;
#pragma unroll
  for (int k = 0; k < QState<GM, NW, D>::KQ; ++k) {
    const int g = wave + NW * k;
    float M = -INFINITY, l = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) qs.o[k][c] = 0.f;
    if (g < G) {
      for (int w = 0; w < nw; ++w) M = fmaxf(M, ml[w * 2 * GM + 2 * g]);
      if (M != -INFINITY) {
        for (int w = 0; w < nw; ++w) {
          const float wt = fast_exp2(ml[w * 2 * GM + 2 * g] - M);
          l += ml[w * 2 * GM + 2 * g + 1] * wt;
#pragma unroll
          for (int c = 0; c < CPL; ++c) qs.o[k][c] += so[w * stride + g * D + lane * CPL + c] * wt;
        }
      }
    }
    qs.M[k] = M;
    qs.l[k] = l;
  }
}

// LDS of selection and finishing.
template <int GM, int NW, int D>
struct SelLds {
  float m[NW][GM], l[NW][GM], lz[GM];
  float best[NW];
  int bj[NW], pick, redo;
  float kv[2][D];      // k*, v* of the evicted row
  float sk[D], sv[D];  // s_k, s_v after this call
  float sq[GM * D];    // S_tilde q (unscaled), query-major
};

// S after the update, staged in LDS for S_tilde q: element (row, col) in 16-byte chunks
// XOR-swizzled by the row, so that the threads of one row (reading chunks p, p + TPR, ...)
// and four neighbouring rows fall into different banks.
template <int D>
__device__ __forceinline__ int s_at(int row, int col) {
  return row * D + ((((col >> 2) ^ ((row & 3) << 2))) << 2) + (col & 3);
}

// Selection and finishing of one KV head by its NW-wave workgroup (see the top of the
// file).  qs: the merged attention state over every row attended to (R with the new
// token); vt / sp / ml: LDS for RW waves to compute the attention again; s_q: the query
// rows in LDS; s_S: LDS for the updated S (D x D floats; it may share the space of vt,
// which is no longer used when S is written).  Everything that does not depend on the
// choice (s_k, s_v, the last row, the first batch of score records) is requested before
// any of it is used, and the summary S with everything that depends only on the choice
// (the evicted row, its logits and its block's running maxima) in one round trip; S is
// held in registers only from there on.
// pre(qs) runs once those first requests are out (the finishing launch combines the
// partial states there).
template <class T, int D, int GM, int NW, int RW, bool ATTN, class Pre>
__device__ __forceinline__ void select_finish(const EvictArgs& e, int head, int old_len, QState<GM, NW, D>& qs,
                              SelLds<GM, NW, D>& sl, typename EvAttn<T, D, GM>::VtTile* vt,
                              typename EvAttn<T, D, GM>::PTile* sp, float* ml, const T* s_q,
                              float* s_S, Pre&& pre) {
  typedef EvAttn<T, D, GM> EA;
  typedef typename EA::FragT FragT;
  constexpr int NT = NW * kWave, KS = D / 32, CPL = D / 64, QRS = EA::QRS;
  constexpr int KQ = QState<GM, NW, D>::KQ;
  constexpr int UB = GM <= 4 ? 16 : (GM <= 8 ? 8 : 4);  // records per thread per batch
  constexpr int SPER = D * D / 4 / NT;                 // float4 entries of S per thread
  constexpr int SCH = SPER < 16 ? SPER : 16;           // of which in registers at a time
  constexpr int NCH = SPER / SCH;
  static_assert(SPER >= 1 && SPER % SCH == 0 && NT % (D / 4) == 0, "S layout");
  static_assert(RW <= NW, "recomputing waves");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool can_append = old_len >= 0 && old_len < e.cap;
  const bool evicts = head_evicts(e, old_len);
  const int G = e.G, ML = e.rec_len, NB = e.rec_len / kEvTB;
  const int n_tok = old_len + 1, last = n_tok - 1;
  const float* rec = e.rec + (size_t)head * (G + 2) * ML;
  T* kc = reinterpret_cast<T*>(e.k_cache) + (size_t)head * e.cap * D;
  T* vc = reinterpret_cast<T*>(e.v_cache) + (size_t)head * e.cap * D;
  float4* Sh = reinterpret_cast<float4*>(e.S + (size_t)head * D * D);

  // requests independent of the choice (S follows with those that depend on it: held
  // in registers only from there on)
  float4 s4[SCH];
  float skv = 0.f, svv = 0.f;
  if (tid < D) {
    skv = e.s_k[(size_t)head * D + tid];
    svv = e.s_v[(size_t)head * D + tid];
  }
  const int ne = e.n_e[head];
  T kl = T(), vl = T();
  if (evicts && tid < D) {
    kl = kc[(size_t)last * D + tid];
    vl = vc[(size_t)last * D + tid];
  }
  float x[UB][GM], y[UB];
  // records of rows base + 4 (tid + NT v) + w (record u = 4 v + w): one 16-byte read per
  // plane and four rows, every read issued and inside the record planes (rec_len is a
  // multiple of 32); rows past n_tok and padded query slots then read as -inf, their
  // norm as +inf.  The masks come after a scheduling barrier, so that all of the reads
  // are out before the first is waited for.
  // Groups of four rows v of the batch at `base` that hold any row below n_tok (the same
  // for every thread): the others are not scored.
  auto groups_in = [&](int base) {
    return min(UB / 4, (n_tok - base + 4 * NT - 1) / (4 * NT));
  };
  auto load_batch = [&](int base) {
    float4 r4[UB / 4][GM + 1];
#pragma unroll
    for (int v = 0; v < UB / 4; ++v) {
      const int jc = min(base + 4 * (tid + NT * v), ML - 4);  // past the planes: rows past n_tok
#pragma unroll
      for (int g = 0; g <= GM; ++g)
        r4[v][g] = *reinterpret_cast<const float4*>(rec + (size_t)(g < GM ? min(g, G - 1) : G) * ML + jc);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int v = 0; v < UB / 4; ++v) {
      const int j0 = base + 4 * (tid + NT * v);
#pragma unroll
      for (int g = 0; g <= GM; ++g) {
        const float rv[4] = {r4[v][g].x, r4[v][g].y, r4[v][g].z, r4[v][g].w};
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const bool ok = j0 + w < n_tok;
          if (g < GM) x[4 * v + w][g] = (ok && g < G) ? rv[w] : -INFINITY;
          else y[4 * v + w] = ok ? rv[w] : INFINITY;
        }
      }
    }
  };
  if (evicts) load_batch(0);
  pre(qs);  // the caller's own requests and work, while these are in flight
  if (tid == 0) sl.redo = 0;

  int js = -1;
  bool s_req = false;  // S requested
  if (evicts) {
    if (tid == 0 && old_len > e.budget) atomicOr(e.flag, 8);  // one eviction cannot reach budget
    const int step = UB * NT;
    const int nb = (n_tok + step - 1) / step;

    if constexpr (ATTN) {
      // log2 Z_g from the merged attention state: it holds the same n_tok base-2 logits
#pragma unroll
      for (int k = 0; k < KQ; ++k) {
        const int g = wave + NW * k;
        if (g < G && lane == 0) sl.lz[g] = qs.M[k] + log2f(qs.l[k]);
      }
      __syncthreads();
    } else {
      // log2 Z_g over the n_tok rows: per batch the thread's max, then its sum (records past
      // n_tok and padded query slots hold -inf and add nothing; no per-record branch)
      float m[GM], l[GM];
#pragma unroll
      for (int g = 0; g < GM; ++g) { m[g] = -INFINITY; l[g] = 0.f; }
      for (int b = 0; b < nb; ++b) {
        if (b > 0) load_batch(b * step);
        const int nv = groups_in(b * step);
#pragma unroll
        for (int g = 0; g < GM; ++g) {
          float mn = m[g];
#pragma unroll
          for (int u = 0; u < UB; ++u)
            if (u / 4 < nv) mn = fmaxf(mn, x[u][g]);
          const float base = mn == -INFINITY ? 0.f : mn;
          float sum = 0.f;
#pragma unroll
          for (int u = 0; u < UB; ++u)
            if (u / 4 < nv) sum += fast_exp2(x[u][g] - base);
          l[g] = l[g] * fast_exp2(m[g] - base) + sum;
          m[g] = mn;
        }
      }
#pragma unroll
      for (int g = 0; g < GM; ++g) {
        if (g < G) {
          const float M = wave_max(m[g]);
          const float ls = wave_sum(M == -INFINITY ? 0.f : l[g] * fast_exp2(m[g] - M));
          if (lane == 0) { sl.m[wave][g] = M; sl.l[wave][g] = ls; }
        }
      }
      __syncthreads();
      if (tid < G) {
        float M = -INFINITY, L = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) M = fmaxf(M, sl.m[w][tid]);
#pragma unroll
        for (int w = 0; w < NW; ++w)
          if (sl.m[w][tid] != -INFINITY) L += sl.l[w][tid] * fast_exp2(sl.m[w][tid] - M);
        sl.lz[tid] = M + log2f(L);
      }
      __syncthreads();
    }

    // S does not depend on the choice: with all of it in one register chunk, it is
    // requested here and arrives while the scores are compared
    if (NCH == 1) {
#pragma unroll
      for (int u = 0; u < SCH; ++u) s4[u] = Sh[tid + NT * u];
      s_req = true;
    }

    // argmin over rows of log2(mean_g alpha_gj) + log2 ||r_j||, lowest row on ties
    float lz[GM];
#pragma unroll
    for (int g = 0; g < GM; ++g) lz[g] = g < G ? sl.lz[g] : 0.f;
    const float log2_g = log2f((float)G);
    float best = INFINITY;
    int bj = INT_MAX;
    for (int b = 0; b < nb; ++b) {
      if (nb > 1) load_batch(b * step);  // one batch: still in registers
      const int nv = groups_in(b * step);
#pragma unroll
      for (int u = 0; u < UB; ++u) {
        if (u / 4 >= nv) continue;
        const int j = b * step + 4 * (tid + NT * (u / 4)) + (u % 4);
        float mx = -INFINITY;
#pragma unroll
        for (int g = 0; g < GM; ++g) mx = fmaxf(mx, x[u][g] - lz[g]);  // -inf past G
        float sm = 0.f;
#pragma unroll
        for (int g = 0; g < GM; ++g) sm += fast_exp2(x[u][g] - lz[g] - mx);
        const float sc = mx + log2f(sm) - log2_g + y[u];
        const bool better = j < n_tok && sc < best;  // rows rise along a thread
        best = better ? sc : best;
        bj = better ? j : bj;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float ob = __shfl_xor(best, off);
      const int oj = __shfl_xor(bj, off);
      if (ob < best || (ob == best && oj < bj)) { best = ob; bj = oj; }
    }
    if (lane == 0) { sl.best[wave] = best; sl.bj[wave] = bj; }
    __syncthreads();
    if (tid == 0) {
      float bb = sl.best[0];
      int j = sl.bj[0];
#pragma unroll
      for (int w = 1; w < NW; ++w)
        if (sl.best[w] < bb || (sl.best[w] == bb && sl.bj[w] < j)) { bb = sl.best[w]; j = sl.bj[w]; }
      sl.pick = j;
    }
    __syncthreads();
    js = __builtin_amdgcn_readfirstlane(sl.pick);
    if (js < 0 || js >= n_tok) js = -1;  // no comparable score (non-finite inputs)
  }

  // requests that depend on the choice: S (to be updated, or for S_tilde q), the evicted
  // row, and per query handled here its logit and its block's running max
  if (!s_req && (ATTN || js >= 0 || e.order >= 1)) {
#pragma unroll
    for (int u = 0; u < SCH; ++u) s4[u] = Sh[tid + NT * u];
  }
  float kf = 0.f, vf = 0.f, xj[KQ], mbj[KQ];
  if (js >= 0) {
    if (tid < D) {
      kf = to_f<T>(kc[(size_t)js * D + tid]);
      vf = to_f<T>(vc[(size_t)js * D + tid]);
    }
    if constexpr (ATTN) {
      const float* bmr = e.blkm + (size_t)head * (G + 1) * NB;
#pragma unroll
      for (int k = 0; k < KQ; ++k) {
        const int g = min(wave + NW * k, G - 1);
        xj[k] = rec[(size_t)g * ML + js];
        mbj[k] = bmr[g * NB + js / kEvTB];
      }
    }
  }

  // bookkeeping: the rank-one update of the vectors and the move of the last row into
  // slot js, or the length and flags of a call that evicts nothing
  if (js >= 0) {
    if (tid < D) {
      sl.kv[0][tid] = kf;
      sl.kv[1][tid] = vf;
      if (js != last) {
        kc[(size_t)js * D + tid] = kl;
        vc[(size_t)js * D + tid] = vl;
      }
      skv += kf;
      svv += vf;
      e.s_k[(size_t)head * D + tid] = skv;
      e.s_v[(size_t)head * D + tid] = svv;
    }
    if (tid == 0) {
      e.n_e[head] = ne + 1;
      e.lens[head] = last;
      if (e.evicted) e.evicted[head] = js;
    }
  } else if (tid == 0) {
    if (evicts) {  // no finite score: keep every row
      atomicOr(e.flag, 4);
      e.lens[head] = n_tok;
    } else if (!can_append) {
      atomicOr(e.flag, 1);
    } else {
      if (old_len + 1 > e.max_len) atomicOr(e.flag, 2);
      e.lens[head] = old_len + 1;
    }
    if (e.evicted) e.evicted[head] = -1;
  }
  if (tid < D) {
    sl.sk[tid] = skv;
    sl.sv[tid] = svv;
  }
  const int ne2 = js >= 0 ? ne + 1 : ne;
  __syncthreads();

  // The evicted row's term leaves the attention state as it was accumulated: p taken at
  // its block's running max mb, scaled to the merged max M (the sum holds p in fp32, the
  // output p rounded to the element type).
  if (ATTN && js >= 0) {
#pragma unroll
    for (int k = 0; k < KQ; ++k) {
      const int g = wave + NW * k;
      if (g < G) {
        const float pj = fast_exp2(xj[k] - mbj[k]);
        if (pj > 0.f) {
          const float s = fast_exp2(mbj[k] - qs.M[k]);
          const float pl = pj * s, po = EA::p_held(pj) * s;
          const float l2 = qs.l[k] - pl;
#pragma unroll
          for (int c = 0; c < CPL; ++c) qs.o[k][c] = fmaf(-po, sl.kv[1][lane * CPL + c], qs.o[k][c]);
          qs.l[k] = l2;
          if (!(kRedoRatio * l2 >= pl) && lane == 0) sl.redo = 1;
        }
      }
    }
  }
  __syncthreads();

  // the attention over the new cache (its rows [0, n)) with RW waves: again, when a
  // removal left too little of some query's sum; without ATTN (no state yet) always
  if (!ATTN || __builtin_amdgcn_readfirstlane(sl.redo)) {
    const int n = js >= 0 ? last
                          : (evicts ? n_tok : (can_append ? old_len + 1 : min(max(old_len, 0), e.cap)));
    const float c2 = e.scale * kLog2e;
    const int r16 = lane & 15, q4 = lane >> 4;
    if (wave < RW) {
      EA at;
      at.init();
      for (int j0 = kEvTB * wave; j0 < n; j0 += kEvTB * RW) {
        FragT kf2[2][KS], vf2[2][KS];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int j = min(j0 + 2 * r16 + hh, n - 1);
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            kf2[hh][ks] = load_frag(kc + (size_t)j * D + 32 * ks + 8 * q4);
            vf2[hh][ks] = load_frag(vc + (size_t)j * D + 32 * ks + 8 * q4);
          }
        }
        f32x4 xl[2];
        EA::logits(s_q, kf2, c2, lane, xl);
        at.block(xl, vf2, j0, n, G, lane, vt[wave], sp[wave]);
      }
      wave_lds_order();
      at.store_lds(reinterpret_cast<float*>(&vt[wave][0][0]), ml + wave * 2 * GM, G, lane);
    }
    __syncthreads();
    merge_waves<GM, NW, D>(qs, reinterpret_cast<const float*>(&vt[0][0][0]),
                           (int)(sizeof(typename EA::VtTile) / sizeof(float)), ml, RW, G, wave, lane);
    __syncthreads();  // vt is read before s_S (which may share its space) is written
  }

  // S after the update S += v* k*^T: written back, and staged in LDS
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    if (ch > 0) {
#pragma unroll
      for (int u = 0; u < SCH; ++u) s4[u] = Sh[tid + NT * (ch * SCH + u)];
    }
#pragma unroll
    for (int u = 0; u < SCH; ++u) {
      const int idx = tid + NT * (ch * SCH + u);
      const int row = idx / (D / 4), c4 = 4 * (idx % (D / 4));
      if (js >= 0) {
        const float va = sl.kv[1][row];
        s4[u].x = fmaf(va, sl.kv[0][c4], s4[u].x);
        s4[u].y = fmaf(va, sl.kv[0][c4 + 1], s4[u].y);
        s4[u].z = fmaf(va, sl.kv[0][c4 + 2], s4[u].z);
        s4[u].w = fmaf(va, sl.kv[0][c4 + 3], s4[u].w);
        Sh[idx] = s4[u];
      }
      *reinterpret_cast<float4*>(&s_S[s_at<D>(row, c4)]) = s4[u];
    }
  }
  __syncthreads();

  // S_tilde q = (S - s_v s_k^T / n_e) q with entries below tau set to zero.  Thread
  // (r, p) takes rows r, r + NT / TPR, ... and the column chunks 4 (p + TPR c); its chunks'
  // s_k / n_e and query entries stay in registers over its rows (queries GB at a time),
  // and the TPR neighbouring lanes of a row add their sums.
  const bool use_sq = e.order >= 1 && ne2 > 0;
  if (use_sq) {
    constexpr int TPR = 8, RPP = NT / TPR, RPT = D / RPP, CPT = D / (4 * TPR);
    constexpr int GB = GM < 4 ? GM : 4;
    static_assert(NT % TPR == 0 && D % RPP == 0 && CPT >= 1 && GM % GB == 0, "S_tilde q layout");
    const float inv_n = 1.f / (float)ne2;
    const int r0 = tid / TPR, part = tid % TPR;
    float skn[CPT][4];
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const float4 sk4 = *reinterpret_cast<const float4*>(&sl.sk[4 * (part + TPR * c)]);
      skn[c][0] = sk4.x * inv_n;
      skn[c][1] = sk4.y * inv_n;
      skn[c][2] = sk4.z * inv_n;
      skn[c][3] = sk4.w * inv_n;
    }
#pragma unroll
    for (int g0 = 0; g0 < GM; g0 += GB) {
      if (g0 < G) {
        float qv[GB][CPT][4];
#pragma unroll
        for (int gi = 0; gi < GB; ++gi)
#pragma unroll
          for (int c = 0; c < CPT; ++c) {
            const T* qg = s_q + min(g0 + gi, G - 1) * QRS + 4 * (part + TPR * c);
            float f[4];
            if constexpr (sizeof(T) == 2) {  // four bf16 in one 8-byte read
              const uint2 w = *reinterpret_cast<const uint2*>(qg);
              f[0] = __uint_as_float(w.x << 16);
              f[1] = __uint_as_float(w.x & 0xffff0000u);
              f[2] = __uint_as_float(w.y << 16);
              f[3] = __uint_as_float(w.y & 0xffff0000u);
            } else {
              const float4 w = *reinterpret_cast<const float4*>(qg);
              f[0] = w.x; f[1] = w.y; f[2] = w.z; f[3] = w.w;
            }
#pragma unroll
            for (int x = 0; x < 4; ++x) qv[gi][c][x] = g0 + gi < G ? f[x] : 0.f;
          }
#pragma unroll
        for (int k = 0; k < RPT; ++k) {
          const int row = r0 + RPP * k;
          const float sr = sl.sv[row];
          float acc[GB];
#pragma unroll
          for (int gi = 0; gi < GB; ++gi) acc[gi] = 0.f;
#pragma unroll
          for (int c = 0; c < CPT; ++c) {
            const float4 s4v = *reinterpret_cast<const float4*>(&s_S[s_at<D>(row, 4 * (part + TPR * c))]);
            float st[4] = {s4v.x - sr * skn[c][0], s4v.y - sr * skn[c][1], s4v.z - sr * skn[c][2],
                           s4v.w - sr * skn[c][3]};
#pragma unroll
            for (int x = 0; x < 4; ++x) st[x] = fabsf(st[x]) < e.tau ? 0.f : st[x];
#pragma unroll
            for (int gi = 0; gi < GB; ++gi)
#pragma unroll
              for (int x = 0; x < 4; ++x) acc[gi] = fmaf(st[x], qv[gi][c][x], acc[gi]);
          }
#pragma unroll
          for (int gi = 0; gi < GB; ++gi) {
            float a = acc[gi];
            a += dpp_f<0xB1>(a);   // quad_perm [1,0,3,2]
            a += dpp_f<0x4E>(a);   // quad_perm [2,3,0,1]
            a += dpp_f<0x141>(a);  // row_half_mirror: the other quad of the eight lanes
            if (part == 0 && g0 + gi < G) sl.sq[(g0 + gi) * D + row] = a;
          }
        }
      }
    }
  }
  __syncthreads();

  // outputs: f_R mixed with f_E_hat = v_bar + scale / n_e * S_tilde q by the Jensen weight
  const int ne_c = e.order < 0 ? 0 : ne2;  // no correction: the output is f_R
  const float inv_c = ne_c > 0 ? 1.f / (float)ne_c : 0.f;
#pragma unroll
  for (int k = 0; k < KQ; ++k) {
    const int g = wave + NW * k;
    if (g < G) {
      const int col = lane * CPL;
      float dot_s = 0.f;
#pragma unroll
      for (int c = 0; c < CPL; ++c) dot_s += to_f<T>(s_q[g * QRS + col + c]) * sl.sk[col + c];
      dot_s = wave_sum(dot_s);
      const float M = qs.M[k], l = qs.l[k];
      const float log_zr = (l > 0.f) ? (M + __log2f(l)) * kLn2 : -INFINITY;
      float w_r = 1.f;
      if (ne_c > 0) {
        const float log_ze = logf((float)ne_c) + e.scale * dot_s / (float)ne_c;  // Jensen estimate
        const float hi = fmaxf(log_zr, log_ze);
        const float lse = hi + logf(expf(log_zr - hi) + expf(log_ze - hi));
        w_r = expf(log_zr - lse);
      }
      T* out = reinterpret_cast<T*>(e.out) + ((size_t)head * G + g) * D + col;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const float f_r = (l > 0.f) ? qs.o[k][c] / l : 0.f;
        float res = f_r;
        if (ne_c > 0) {
          float fe = sl.sv[col + c] * inv_c;
          if (e.order >= 1) fe += e.scale * inv_c * sl.sq[g * D + col + c];
          res = w_r * f_r + (1.f - w_r) * fe;
        }
        out[c] = from_f<T>(res);
      }
      if (lane == 0) {
        const size_t pair = (size_t)head * G + g;
        if (e.lse_out) e.lse_out[pair] = log_zr;
        if (e.w_r_out) e.w_r_out[pair] = w_r;
      }
    }
  }
}

// Waves per scoring workgroup: with the attention, as many as the LDS holds next to
// S_tilde (one workgroup per CU); scoring alone, four (two workgroups per CU).
template <class T, int GM, bool ATTN>
constexpr int ev_waves() {
  return !ATTN ? 4 : (sizeof(T) == 2 ? (GM <= 4 ? 8 : 4) : (GM <= 4 ? 4 : 2));
}

template <class T, int D, int GM, int NW, bool ATTN> struct EvLds;
template <class T, int D, int GM, int NW> struct EvLds<T, D, GM, NW, true> {
  typedef EvAttn<T, D, GM> EA;
  SumLds<T, D> sm;             // S_tilde of the head being scored
  typename EA::VtTile vt[NW];  // per wave; after a segment, the wave's o rows
  typename EA::PTile sp[NW];
  T q[16 * EA::QRS];
  float vinit[D];             // s_v / scale: the start of the S_tilde k accumulators
  float ml[NW * 2 * GM];
};
template <class T, int D, int GM, int NW> struct EvLds<T, D, GM, NW, false> {
  typedef EvAttn<T, D, GM> EA;
  SumLds<T, D> sm;
  T q[16 * EA::QRS];
  float vinit[D];             // s_v / scale: the start of the S_tilde k accumulators
  SelLds<GM, NW, D> sel;
};

template <class T, int D, int GM>
struct FinLds {
  typedef EvAttn<T, D, GM> EA;
  struct Redo {
    typename EA::VtTile vt[kFinWaves];
    typename EA::PTile sp[kFinWaves];
  };
  union {
    Redo r;          // an attention computed again
    float S[D * D];  // then the updated S
  } u;
  T q[16 * EA::QRS];
  float ml[kFinWaves * 2 * GM];
  SelLds<GM, kFinWaves, D> sel;
};

// The scoring workgroup that holds block b of the flattened (head, 32-row block) range:
// workgroup w takes blocks [w N / nwg, (w + 1) N / nwg), N = n_heads * hblocks.
__device__ __forceinline__ int wg_of_block(const EvictArgs& e, int64_t b) {
  const int64_t nblk = (int64_t)e.n_heads * e.hblocks;
  return (int)(((b + 1) * e.nwg - 1) / nblk);
}

// Blocks [s0, s1) of one head by the NW-wave workgroup (see the top of the file).  With
// ATTN the rows are scored and attended to, and the merged state is written as the
// head's partial `slot`; without, a head that evicts is scored, and the workgroup (which
// then holds the whole head) selects, updates and attends to the new cache at the end.
template <class T, int D, int GM, int NW, bool ATTN>
__device__ __forceinline__ void ev_segment(const EvictArgs& e, EvLds<T, D, GM, NW, ATTN>& L, int head,
                                           int s0, int s1, int slot) {
  typedef EvAttn<T, D, GM> EA;
  typedef typename EA::FragT FragT;
  constexpr int KS = D / 32;   // contraction steps; also 8-dim groups per lane and row
  constexpr int NTI = D / 16;  // 16-row tiles of S_tilde k
  constexpr int NT = NW * kWave;
  constexpr int CPL = D / 64;
  // the wave index, lengths and loop bounds are the same for all lanes; held in scalar
  // registers, they make the loops below uniform control flow rather than per-lane loops
  const int tid = tid_here();
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q4 = lane >> 4, r16 = lane & 15;
  const int G = e.G, hb = e.hblocks;
  const int ML = e.rec_len, NB = e.rec_len / kEvTB;
  const float c2 = e.scale * kLog2e;

  const int old_len = __builtin_amdgcn_readfirstlane(e.lens[head]);
  const bool can_append = old_len >= 0 && old_len < e.cap;
  const bool evicts = head_evicts(e, old_len);
  // rows attended to: R with the new token (the whole cache when there is no room);
  // scored alone: R when the head evicts, nothing otherwise
  const int n_rows = !ATTN ? (evicts ? old_len + 1 : 0)
                           : (can_append ? old_len + 1 : min(max(old_len, 0), e.cap));
  const int t0 = kEvTB * s0;  // below max_len <= cap
  const int t1 = s1 == hb ? n_rows : min(kEvTB * s1, n_rows);
  // the workgroup whose blocks hold the new row appends it (the head's last block for
  // rows past them); nothing reads that cache row before the segment's rows are read (the
  // new token is read from k_new / v_new), so the copy is written after them: with the
  // attention, read then as well (no registers held over the loop); scoring alone, read
  // here (the workgroup then waits for nothing but its own rows)
  const int nb_new = min(old_len / kEvTB, hb - 1);
  const bool appends = can_append && wave == 0 && nb_new >= s0 && nb_new < s1;
  uint4 new_piece = make_uint4(0, 0, 0, 0);
  if (!ATTN && appends) new_piece = append_read<T, D>(e, head, lane);

  if (ATTN || t0 < t1) {  // uniform
    const T* kc = reinterpret_cast<const T*>(e.k_cache) + (size_t)head * e.cap * D;
    const T* vc = reinterpret_cast<const T*>(e.v_cache) + (size_t)head * e.cap * D;
    const T* kn = reinterpret_cast<const T*>(e.k_new) + (size_t)head * D;
    const T* vn = reinterpret_cast<const T*>(e.v_new) + (size_t)head * D;
    float* rec = e.rec + (size_t)head * (G + 2) * ML;
    float* bmr = e.blkm + (size_t)head * (G + 1) * NB;

    // rows j0 + 2 (l % 16) + hh; rows past t1 read the last row again (masked in the
    // attention; their records land in the padding of the record rows): every lane
    // issues every load, so the compiler can count the loads in flight and waits for one
    // block while the next is still arriving
    const int jmax = max(t1 - 1, t0);  // a cache row even for an empty segment
    auto load = [&](FragT (&kf)[2][KS], FragT (&vf)[2][KS], int j0) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int j = min(j0 + 2 * r16 + hh, jmax);
        const bool nw = can_append && j == old_len;
        const T* kr = nw ? kn : kc + (size_t)j * D;
        const T* vr = nw ? vn : vc + (size_t)j * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          kf[hh][ks] = load_frag(kr + 32 * ks + 8 * q4);
          vf[hh][ks] = load_frag(vr + 32 * ks + 8 * q4);
        }
      }
    };
    FragT ka[2][KS], va[2][KS], kb[2][KS], vb[2][KS];
    int j0 = t0 + kEvTB * wave;
    load(ka, va, j0);  // in flight while the summary is formed

    QueryRows<T, D, NT> qr;
    qr.load(e, head);
    const float svv = tid < D ? e.s_v[(size_t)head * D + tid] : 0.f;
    const int ne = evicts ? build_summary<T, D, NT>(e, head, L.sm) : e.n_e[head];
    qr.store(L.q);
    // r_j = v_j - cf (v_bar / cf + S_tilde k_j): the accumulators of S_tilde k_j start at
    // v_bar / cf = s_v / scale, so the mean comes out of the MFMAs
    const float cf = ne > 0 ? e.scale / (float)ne : 0.f;
    if (tid < D) L.vinit[tid] = ne > 0 ? svv / e.scale : 0.f;
    __syncthreads();  // S_tilde, v_bar and the queries are in LDS

    EA at;
    at.init();
    auto process = [&](const FragT (&kf)[2][KS], const FragT (&vf)[2][KS], int j0) {
      f32x4 x[2];
      EA::logits(L.q, kf, c2, lane, x);
      // scoring records; every lane stores (no branch around a store): a head that does
      // not evict writes into the first columns of the spare plane G + 1
      const int col = evicts ? j0 + 2 * r16 : 2 * r16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int g = 4 * q4 + i;
        *reinterpret_cast<float2*>(&rec[(size_t)((evicts && g < G) ? g : G + 1) * ML + col]) =
            make_float2(x[0][i], x[1][i]);
      }
      float rr[2] = {1.f, 1.f};
      if (evicts) {
        // S_tilde k: tile t = 2c + s holds dims 32c + 8 (lane/16) + 4s + i in lane rows
        // 4 (lane/16) + i, i.e. element 4s + i of the lane's V fragment c.
        rr[0] = rr[1] = 0.f;
#pragma unroll
        for (int t = 0; t < NTI; ++t) {
          const int c = t >> 1, s = t & 1;
          const int row = 32 * c + 8 * (r16 >> 2) + 4 * s + (r16 & 3);
          const float4 vb4 = *reinterpret_cast<const float4*>(&L.vinit[32 * c + 8 * q4 + 4 * s]);
          f32x4 ta[2];
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            ta[hh][0] = vb4.x;
            ta[hh][1] = vb4.y;
            ta[hh][2] = vb4.z;
            ta[hh][3] = vb4.w;
          }
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            if constexpr (sizeof(T) == 2) {
              const int a = SumLds<T, D>::at(row, 32 * ks + 8 * q4);
              const bf16x8 ah = lds_frag(&L.sm.hi[a]);
              const bf16x8 al = lds_frag(&L.sm.lo[a]);
#pragma unroll
              for (int hh = 0; hh < 2; ++hh) {
                mma(ta[hh], ah, kf[hh][ks]);
                mma(ta[hh], al, kf[hh][ks]);
              }
            } else {
              const f32x8 af = lds_frag(&L.sm.st[SumLds<T, D>::at(row, 32 * ks + 8 * q4)]);
#pragma unroll
              for (int hh = 0; hh < 2; ++hh) mma(ta[hh], af, kf[hh][ks]);
            }
          }
#pragma unroll
          for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float r = fmaf(-cf, ta[hh][i], elem_f(vf[hh][c], 4 * s + i));
              rr[hh] = fmaf(r, r, rr[hh]);
            }
          // one tile's LDS reads in flight at a time: hoisting all of them would not fit
          __builtin_amdgcn_sched_barrier(0);
        }
        rr[0] = cross_row_sum(rr[0]);
        rr[1] = cross_row_sum(rr[1]);
      }
      *reinterpret_cast<float2*>(&rec[(size_t)(evicts ? G : G + 1) * ML + col]) =
          make_float2(0.5f * log2f(rr[0]), 0.5f * log2f(rr[1]));  // the same from four lanes
      if constexpr (ATTN) {
        at.block(x, vf, j0, t1, G, lane, L.vt[wave], L.sp[wave]);
        // the running max of query 4 (l / 16) + (l % 4) after this block
        const int gm = 4 * q4 + (lane & 3);
        bmr[((evicts && gm < G) ? gm : G) * NB + (evicts ? j0 / kEvTB : 0)] = at.m_of_lane(lane);
      }
    };

    // 32-row blocks j0, j0 + 32 NW, ... of this wave; the next block's rows are requested
    // before the current block is processed (two register sets)
    for (; j0 < t1; j0 += 2 * NW * kEvTB) {
      load(kb, vb, j0 + NW * kEvTB);
      process(ka, va, j0);
      if (j0 + NW * kEvTB >= t1) break;
      load(ka, va, j0 + 2 * NW * kEvTB);
      process(kb, vb, j0 + NW * kEvTB);
    }

    if constexpr (ATTN) {
      // the waves' states, merged per query, as the head's partial `slot`
      wave_lds_order();
      at.store_lds(reinterpret_cast<float*>(&L.vt[wave][0][0]), L.ml + wave * 2 * GM, G, lane);
      __syncthreads();
      QState<GM, NW, D> qs;
      merge_waves<GM, NW, D>(qs, reinterpret_cast<const float*>(&L.vt[0][0][0]),
                             (int)(sizeof(typename EA::VtTile) / sizeof(float)), L.ml, NW, G, wave, lane);
#pragma unroll
      for (int k = 0; k < QState<GM, NW, D>::KQ; ++k) {
        const int g = wave + NW * k;
        if (g < G) {
          const size_t pb = ((size_t)head * e.maxslots + slot) * G + g;
#pragma unroll
          for (int c = 0; c < CPL; ++c) e.part_o[pb * D + lane * CPL + c] = qs.o[k][c];
          if (lane == 0) {
            e.part_ml[pb * 2] = qs.M[k];
            e.part_ml[pb * 2 + 1] = qs.l[k];
          }
        }
      }
    }
  }
  if (appends) {
    if constexpr (ATTN) append_new_row<T, D>(e, head, old_len, lane);
    else append_write<T, D>(e, head, old_len, lane, new_piece);
  }
  if constexpr (!ATTN) {
    // The workgroup holds the whole head: its records and the appended row are visible
    // to all of its waves after a barrier, and it selects, updates, then attends to the
    // new cache itself (rows it has just read, mostly from L2), with its V tiles where
    // S_tilde was; no second launch.
    typedef typename EA::VtTile VtT;
    typedef typename EA::PTile PtT;
    constexpr int RW0 = (int)((sizeof(SumLds<T, D>) - NW * 2 * GM * sizeof(float)) / (sizeof(VtT) + sizeof(PtT)));
    constexpr int RW = RW0 < NW ? RW0 : NW;  // waves that attend (as many as the space holds)
    static_assert(RW >= 1, "V tiles fit in place of S_tilde");
    static_assert(sizeof(SumLds<T, D>) >= D * D * sizeof(float), "S fits in place of S_tilde");
    char* base = reinterpret_cast<char*>(&L.sm);
    VtT* vt = reinterpret_cast<VtT*>(base);
    PtT* sp = reinterpret_cast<PtT*>(base + RW * sizeof(VtT));
    float* ml = reinterpret_cast<float*>(base + RW * (sizeof(VtT) + sizeof(PtT)));
    if (t0 >= t1) {  // a head that does not evict: its queries, for the attention
      QueryRows<T, D, NT> qr;
      qr.load(e, head);
      qr.store(L.q);
    }
    __syncthreads();
    QState<GM, NW, D> qs;
    select_finish<T, D, GM, NW, RW, false>(e, head, old_len, qs, L.sel, vt, sp, ml, L.q,
                                           reinterpret_cast<float*>(&L.sm),
                                           [](QState<GM, NW, D>&) {});
  }
}

}  // namespace

// Scoring pass.  With the attention (ATTN): nwg workgroups (about one per CU) take equal,
// contiguous shares of the flattened (head, 32-row block) range, so heads of any length
// spread evenly over the CUs; a share crosses into at most a few heads, each a segment
// (queries and S_tilde formed per segment), whose merged state is written as the head's
// partial number w - (first workgroup of the head).  The head's last block also takes
// rows past hblocks * 32 (a cache longer than max_len after a full call).  Scoring alone:
// one workgroup per head, which also selects, updates and then attends to the new cache.
template <class T, int D, int GM, int NW, bool ATTN>
__global__ void __launch_bounds__(NW * kWave, ATTN ? 1 : 2) k_evict_attn(EvictArgs e) {
  typedef EvLds<T, D, GM, NW, ATTN> LT;
  static_assert(sizeof(LT) <= 160 * 1024, "LDS of the scoring workgroup");
  __shared__ __align__(16) LT L;
  if constexpr (ATTN) {
    const int hb = e.hblocks;
    const int64_t nblk = (int64_t)e.n_heads * hb;
    const int64_t b0 = (int64_t)blockIdx.x * nblk / e.nwg, b1 = (int64_t)(blockIdx.x + 1) * nblk / e.nwg;
    for (int head = (int)(b0 / hb); b1 > b0 && (int64_t)head * hb < b1; ++head) {
      const int s0 = (int)max(b0 - (int64_t)head * hb, (int64_t)0);
      const int s1 = (int)min(b1 - (int64_t)head * hb, (int64_t)hb);
      __syncthreads();  // the previous segment's reads of the LDS are done
      ev_segment<T, D, GM, NW, true>(e, L, head, s0, s1, blockIdx.x - wg_of_block(e, (int64_t)head * hb));
    }
  } else {
    ev_segment<T, D, GM, NW, false>(e, L, blockIdx.x, 0, e.hblocks, 0);
  }
}

// Finishing launch, one 4-wave workgroup per KV head (two fit on a CU for bf16): the head's
// partial states combined in order, then selection, update and correction.
template <class T, int D, int GM>
__global__ void __launch_bounds__(kFinWaves * kWave, 2) k_evict_finish(EvictArgs e) {
  typedef FinLds<T, D, GM> LT;
  constexpr int NT = kFinWaves * kWave, CPL = D / 64, SUB = 8;
  static_assert(sizeof(LT) <= 160 * 1024, "LDS of the finishing workgroup");
  static_assert(sizeof(T) == 4 || sizeof(LT) <= 80 * 1024, "two bf16 finishing workgroups per CU");
  __shared__ __align__(16) LT L;
  const int head = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int old_len = __builtin_amdgcn_readfirstlane(e.lens[head]);
  const int G = e.G;
  const int hb = e.hblocks;
  const int ns = wg_of_block(e, (int64_t)(head + 1) * hb - 1) - wg_of_block(e, (int64_t)head * hb) + 1;

  QueryRows<T, D, NT> qr;
  qr.load(e, head);
  // the partial states per query, combined in order once the selection's first requests
  // are out; every load is issued before the first is used (partial indices clamped to
  // the count)
  auto combine = [&](QState<GM, kFinWaves, D>& qs) {
#pragma unroll
    for (int k = 0; k < QState<GM, kFinWaves, D>::KQ; ++k) {
      const int g = min(wave + kFinWaves * k, G - 1);  // waves past G: loads never used
      const size_t base = (size_t)head * e.maxslots;
      auto o_at = [&](int s, int c) {
        return e.part_o + ((base + min(s, ns - 1)) * G + g) * D + lane * CPL + c;
      };
      const float2 ml = *reinterpret_cast<const float2*>(e.part_ml + ((base + min(lane, ns - 1)) * G + g) * 2);
      float ov[SUB][CPL];
#pragma unroll
      for (int u = 0; u < SUB; ++u)
#pragma unroll
        for (int c = 0; c < CPL; ++c) ov[u][c] = *o_at(u, c);
      const bool live = lane < ns;
      const float M = wave_max(live ? ml.x : -INFINITY);
      const float w = (live && M != -INFINITY) ? fast_exp2(ml.x - M) : 0.f;
      qs.M[k] = M;
      qs.l[k] = wave_sum(live ? ml.y * w : 0.f);
      float o[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) o[c] = 0.f;
      for (int s0 = 0; s0 < ns; s0 += SUB) {
        if (s0 > 0) {
#pragma unroll
          for (int u = 0; u < SUB; ++u)
#pragma unroll
            for (int c = 0; c < CPL; ++c) ov[u][c] = *o_at(s0 + u, c);
        }
#pragma unroll
        for (int u = 0; u < SUB; ++u) {
          if (s0 + u < ns) {
            const float wu = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), s0 + u));
#pragma unroll
            for (int c = 0; c < CPL; ++c) o[c] = fmaf(wu, ov[u][c], o[c]);
          }
        }
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) qs.o[k][c] = o[c];
    }
    qr.store(L.q);  // read after the selection's barriers
  };
  QState<GM, kFinWaves, D> qs;
  select_finish<T, D, GM, kFinWaves, kFinWaves, true>(e, head, old_len, qs, L.sel, L.u.r.vt,
                                                      L.u.r.sp, L.ml, L.q, L.u.S, combine);
}

int evict_waves(bool bf16, int G) {
  if (bf16) return G <= 4 ? ev_waves<bf16_t, 4, true>() : ev_waves<bf16_t, 16, true>();
  return G <= 4 ? ev_waves<float, 4, true>() : ev_waves<float, 16, true>();
}

int evict_max_slices() { return kMaxSlices; }

template <class T, int D, int GM>
static hipError_t launch_evict_g(const EvictArgs& e, hipStream_t st) {
  if (e.fused) {
    constexpr int NW = ev_waves<T, GM, true>();
    hipLaunchKernelGGL((k_evict_attn<T, D, GM, NW, true>), dim3(e.nwg), dim3(NW * kWave), 0, st, e);
    hipLaunchKernelGGL((k_evict_finish<T, D, GM>), dim3(e.n_heads), dim3(kFinWaves * kWave), 0, st, e);
  } else {
    constexpr int NW = ev_waves<T, GM, false>();
    hipLaunchKernelGGL((k_evict_attn<T, D, GM, NW, false>), dim3(e.n_heads), dim3(NW * kWave), 0, st, e);
  }
  return hipGetLastError();
}

template <class T, int D>
static hipError_t launch_evict_t(const EvictArgs& e, hipStream_t st) {
  if (e.G <= 4) return launch_evict_g<T, D, 4>(e, st);
  if (e.G <= 8) return launch_evict_g<T, D, 8>(e, st);
  return launch_evict_g<T, D, 16>(e, st);
}

hipError_t launch_evict(const EvictArgs& e, bool bf16, int d, hipStream_t st) {
  if (e.fused && (e.nwg < 1 || e.maxslots < 1 || e.maxslots > kMaxSlices)) return hipErrorInvalidValue;
  if (bf16) return d == 64 ? launch_evict_t<bf16_t, 64>(e, st) : launch_evict_t<bf16_t, 128>(e, st);
  return d == 64 ? launch_evict_t<float, 64>(e, st) : launch_evict_t<float, 128>(e, st);
}

}  // namespace mkv
