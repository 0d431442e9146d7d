// Moment-informed eviction at a decoding step (Algorithm 1 Phase 1), run ahead of the
// corrected attention of Phase 2 (which then goes through the decode launches on the
// updated cache and summary).
//
// k_evict_scores: n_heads x nslice workgroups of 4 waves.  The workgroup first forms the
//   summary's clamped covariance S_tilde = S - s_v s_k^T / n_e (entries below tau set to
//   zero; zero when n_e = 0) from the raw moments into LDS: hi / lo bf16 planes for bf16
//   caches, fp32 otherwise.  Each wave then takes 32-row blocks of the workgroup's rows
//   of R, the new token included (row lens, read from k_new / v_new), and writes for
//   every row j
//     x_gj = scale log2(e) q_g . k_j           (base-2 logits of the G queries)
//     y_j  = log2 ||r_j||,  r_j = v_j - v_bar - (scale / n_e) S_tilde k_j   (Eq. residual)
//   S_tilde k_j runs on MFMA with the same K fragments as the logits (B operand) and
//   S_tilde rows from LDS (A operand).  The rows of each 16-row MFMA tile are taken in
//   the order that leaves every lane holding the products for exactly the dimensions of
//   v_j it loaded (dims 32c + 8 (lane / 16) + e), so r_j and its squared norm are formed
//   in registers and finished with a 4-lane sum.
// k_evict_select: one workgroup per KV head.  log2 Z_g over R from the logits, the
//   group-mean softmax weight alpha_j = mean_g 2^(x_gj - log2 Z_g) in the log domain (so
//   no weight underflows), the argmin of log2 alpha_j + y_j (the lowest row on ties),
//   then the rank-one update n_e += 1, s_k += k*, s_v += v*, S += v* k*^T (App. A.1
//   Eq. app_update) and the move of the last row into the freed one.
#include <climits>

#include "mkv_bf16.h"
#include "mkv_device.h"
#include "mkv_evict.h"

namespace mkv {

namespace {

constexpr int kEvThreads = 256;
constexpr int kEvTB = 32;  // rows per block

// LDS copy of S_tilde with rows padded by 16 bytes.
template <class T, int D> struct SumLds;
template <int D> struct SumLds<bf16_t, D> {
  static constexpr int RS = D + 8;
  bf16_t hi[D * RS];
  bf16_t lo[D * RS];
};
template <int D> struct SumLds<float, D> {
  static constexpr int RS = D + 4;
  float st[D * RS];
};

// bf16 S_tilde rows: 16-byte chunks XOR-swizzled by bit 4 of the row.  The 16 rows one
// MFMA read touches (r + {0..3, 8..11, 16..19, 24..27}) would otherwise fall pairwise
// into the same bank group (rows 16 apart); swizzled, each 16-lane pass of the read
// covers 16 different groups.
template <class T>
__device__ __forceinline__ int scol(int row, int col) {
  if constexpr (sizeof(T) == 2) return col ^ (((row >> 4) & 1) << 5);
  else return col;
}

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

// S_tilde of one head into LDS; every thread handles D*D/8/256 chunks of 8 entries of a
// row (all loads issued before any is used).
template <class T, int D>
__device__ __forceinline__ void build_summary(const EvictArgs& e, int head, SumLds<T, D>& sm) {
  constexpr int PER = D * D / 8 / kEvThreads;
  constexpr int RS = SumLds<T, D>::RS;
  const int tid = threadIdx.x;
  const int c0 = 8 * (tid % (D / 8));
  const int ne = e.n_e[head];
  const float inv_n = ne > 0 ? 1.f / (float)ne : 0.f;
  const float* Sh = e.S + (size_t)head * D * D;
  const f32x8 skc = load_frag(e.s_k + (size_t)head * D + c0);
  f32x8 raw[PER];
  float sv[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int row = (tid + kEvThreads * u) / (D / 8);
    raw[u] = load_frag(Sh + (size_t)row * D + c0);
    sv[u] = e.s_v[(size_t)head * D + row];
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int row = (tid + kEvThreads * u) / (D / 8);
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
      *reinterpret_cast<uint4*>(&sm.hi[row * RS + scol<T>(row, c0)]) = make_uint4(h[0], h[1], h[2], h[3]);
      *reinterpret_cast<uint4*>(&sm.lo[row * RS + scol<T>(row, c0)]) = make_uint4(l[0], l[1], l[2], l[3]);
    } else {
      float4* P = reinterpret_cast<float4*>(&sm.st[row * RS + c0]);
      P[0] = make_float4(st[0], st[1], st[2], st[3]);
      P[1] = make_float4(st[4], st[5], st[6], st[7]);
    }
  }
}

// The new token: wave 0 of the workgroup given the job copies k_new / v_new to cache row
// `row`, 16 bytes per lane.
template <class T, int D>
__device__ __forceinline__ void append_new_row(const EvictArgs& e, int head, int row, int lane) {
  constexpr int NV = D * (int)sizeof(T) / 16;
  if (lane < 2 * NV) {
    const bool is_v = lane >= NV;
    const int piece = lane % NV;
    const uint4* src = reinterpret_cast<const uint4*>(
        reinterpret_cast<const T*>(is_v ? e.v_new : e.k_new) + (size_t)head * D) + piece;
    T* cache = reinterpret_cast<T*>(is_v ? e.v_cache : e.k_cache);
    uint4* dst = reinterpret_cast<uint4*>(cache + ((size_t)head * e.cap + row) * D) + piece;
    *dst = *src;
  }
}

// Whether this call evicts from the head: the new row fits in the cache and in the
// row bound, and the cache then holds more than `budget` rows.
__device__ __forceinline__ bool head_evicts(const EvictArgs& e, int old_len) {
  return old_len >= 0 && old_len < e.cap && old_len + 1 <= e.max_len && old_len + 1 > e.budget;
}

}  // namespace

// Selection (one KV head, NT threads): log2 Z_g over R from the logits, the group-mean
// softmax weight in the log domain, the argmin (lowest row on ties), then the rank-one
// update and the move of the last row.  Everything that does not depend on the choice
// (the summary S, the last row, the score records of up to UB rows per thread) is
// requested before any of it is used, so a short cache costs three round trips to
// memory: the records and S together, then the evicted row.  GM bounds the group size
// G (4, 8 or 16); rows per thread per batch shrink as it grows.  Also handles a head that
// does not evict this call (append only, or the flags).
template <int GM, int NW, int D>
struct SelLds {
  float m[NW][GM], l[NW][GM], lz[GM];
  float best[NW];
  int bj[NW], pick;
  float kv[2][D];
};

template <class T, int D, int GM, int NT>
__device__ __forceinline__ void select_head(const EvictArgs& e, int head, int old_len,
                                            SelLds<GM, NT / kWave, D>& sl) {
  constexpr int NW = NT / kWave;
  constexpr int UB = GM <= 4 ? 8 : (GM <= 8 ? 4 : 2);
  constexpr int SPER = D * D / 4 / NT;  // float4 entries of S per thread
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool can_append = old_len >= 0 && old_len < e.cap;
  if (!head_evicts(e, old_len)) {
    if (tid == 0) {
      if (!can_append) {
        atomicOr(e.flag, 1);
      } else {
        if (old_len + 1 > e.max_len) atomicOr(e.flag, 2);
        e.lens[head] = old_len + 1;
      }
      if (e.evicted) e.evicted[head] = -1;
    }
    return;
  }
  const int n_tok = old_len + 1, last = n_tok - 1;
  const int G = e.G, ML = e.rec_len;
  const float* rec = e.rec + (size_t)head * (G + 2) * ML;
  T* kc = reinterpret_cast<T*>(e.k_cache) + (size_t)head * e.cap * D;
  T* vc = reinterpret_cast<T*>(e.v_cache) + (size_t)head * e.cap * D;
  float4* Sh = reinterpret_cast<float4*>(e.S + (size_t)head * D * D);
  if (tid == 0 && old_len > e.budget) atomicOr(e.flag, 8);  // one eviction cannot reach budget

  // requests independent of the choice
  float4 s4[SPER];
#pragma unroll
  for (int u = 0; u < SPER; ++u) s4[u] = Sh[tid + NT * u];
  T kl = T(), vl = T();
  if (tid < D) {
    kl = kc[(size_t)last * D + tid];
    vl = vc[(size_t)last * D + tid];
  }
  float x[UB][GM], y[UB];
  auto load_batch = [&](int base) {
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int j = base + tid + NT * u;
      const bool ok = j < n_tok;
#pragma unroll
      for (int g = 0; g < GM; ++g) x[u][g] = (ok && g < G) ? rec[(size_t)g * ML + j] : -INFINITY;
      y[u] = ok ? rec[(size_t)G * ML + j] : INFINITY;
    }
  };
  const int step = UB * NT;
  const int nb = (n_tok + step - 1) / step;

  // log2 Z_g over the n_tok rows
  float m[GM], l[GM];
#pragma unroll
  for (int g = 0; g < GM; ++g) { m[g] = -INFINITY; l[g] = 0.f; }
  for (int b = 0; b < nb; ++b) {
    load_batch(b * step);
#pragma unroll
    for (int u = 0; u < UB; ++u)
#pragma unroll
      for (int g = 0; g < GM; ++g) {
        const float mn = fmaxf(m[g], x[u][g]);
        if (mn != -INFINITY) {
          l[g] = l[g] * fast_exp2(m[g] - mn) + fast_exp2(x[u][g] - mn);
          m[g] = mn;
        }
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

  // argmin over rows of log2(mean_g alpha_gj) + log2 ||r_j||, lowest row on ties
  float lz[GM];
#pragma unroll
  for (int g = 0; g < GM; ++g) lz[g] = g < G ? sl.lz[g] : 0.f;
  const float log2_g = log2f((float)G);
  float best = INFINITY;
  int bj = INT_MAX;
  for (int b = 0; b < nb; ++b) {
    if (nb > 1) load_batch(b * step);  // one batch: still in registers
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int j = b * step + tid + NT * u;
      float mx = -INFINITY;
#pragma unroll
      for (int g = 0; g < GM; ++g) mx = fmaxf(mx, g < G ? x[u][g] - lz[g] : -INFINITY);
      float sm = 0.f;
#pragma unroll
      for (int g = 0; g < GM; ++g)
        if (g < G) sm += fast_exp2(x[u][g] - lz[g] - mx);
      const float sc = mx + log2f(sm) - log2_g + y[u];
      if (j < n_tok && sc < best) { best = sc; bj = j; }  // rows rise along a thread
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
  const int js = sl.pick;
  if (js < 0 || js >= n_tok) {  // no comparable score (non-finite inputs): keep every row
    if (tid == 0) {
      atomicOr(e.flag, 4);
      e.lens[head] = n_tok;
      if (e.evicted) e.evicted[head] = -1;
    }
    return;
  }

  // rank-one update and the move of the last row into slot js
  if (tid < D) {
    const T ks = kc[(size_t)js * D + tid], vs = vc[(size_t)js * D + tid];
    const float kf = to_f<T>(ks), vf = to_f<T>(vs);
    sl.kv[0][tid] = kf;
    sl.kv[1][tid] = vf;
    if (js != last) {
      kc[(size_t)js * D + tid] = kl;
      vc[(size_t)js * D + tid] = vl;
    }
    e.s_k[(size_t)head * D + tid] += kf;
    e.s_v[(size_t)head * D + tid] += vf;
  }
  if (tid == 0) {
    e.n_e[head] += 1;
    e.lens[head] = last;
    if (e.evicted) e.evicted[head] = js;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < SPER; ++u) {
    const int idx = tid + NT * u;
    const int row = idx / (D / 4), c = 4 * (idx % (D / 4));
    const float va = sl.kv[1][row];
    s4[u].x = fmaf(va, sl.kv[0][c], s4[u].x);
    s4[u].y = fmaf(va, sl.kv[0][c + 1], s4[u].y);
    s4[u].z = fmaf(va, sl.kv[0][c + 2], s4[u].z);
    s4[u].w = fmaf(va, sl.kv[0][c + 3], s4[u].w);
    Sh[idx] = s4[u];
  }
}

template <class T, int D, int GM>
__global__ void __launch_bounds__(kEvThreads, sizeof(T) == 2 ? 2 : 1) k_evict_scores(EvictArgs e) {
  typedef typename Frag<T>::type FragT;
  constexpr int KS = D / 32;  // contraction steps; also 8-dim groups per lane and row
  constexpr int NT = D / 16;  // 16-row tiles of S_tilde k
  constexpr int RS = SumLds<T, D>::RS;
  __shared__ __align__(16) SumLds<T, D> sm;
  __shared__ __align__(16) float s_vbar[D];
  constexpr int QRS = D + 16 / (int)sizeof(T);  // query rows padded by 16 bytes
  __shared__ __align__(16) T s_q[16 * QRS];
  __shared__ SelLds<GM, kEvThreads / kWave, D> sel;  // the selection, one workgroup per head

  const int head = blockIdx.x / e.nslice, slice = blockIdx.x % e.nslice;
  // the wave index and the length are the same for all lanes; held in scalar registers,
  // they make the block loop below uniform control flow rather than a per-lane loop
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q4 = lane >> 4, r16 = lane & 15;
  const int old_len = __builtin_amdgcn_readfirstlane(e.lens[head]);
  const bool can_append = old_len >= 0 && old_len < e.cap;
  // the workgroup whose rows hold the new one appends it (the last one for rows past them)
  if (can_append && wave == 0 && min(old_len / e.slice_len, e.nslice - 1) == slice)
    append_new_row<T, D>(e, head, old_len, lane);
  const int t0 = slice * e.slice_len;
  const int t1 = min(t0 + e.slice_len, old_len + 1);
  if (!head_evicts(e, old_len) || t0 >= t1) {  // uniform over the workgroup
    if (e.nslice == 1) select_head<T, D, GM, kEvThreads>(e, head, old_len, sel);  // lens, flags
    return;
  }

  const int G = e.G;
  const T* kc = reinterpret_cast<const T*>(e.k_cache) + (size_t)head * e.cap * D;
  const T* vc = reinterpret_cast<const T*>(e.v_cache) + (size_t)head * e.cap * D;
  const T* kn = reinterpret_cast<const T*>(e.k_new) + (size_t)head * D;
  const T* vn = reinterpret_cast<const T*>(e.v_new) + (size_t)head * D;
  const int ML = e.rec_len;  // rows of the record planes (whole 32-row blocks)
  float* rec = e.rec + (size_t)head * (G + 2) * ML;
  const float c2 = e.scale * kLog2e;

  // rows j0 + 16 hh + lane % 16: K and V fragments at dims 32 ks + 8 (lane / 16).  Rows
  // past t1 read row t1 - 1 again (their records land in the padding of the record rows
  // or are never written): every lane issues every load, so the compiler can count the
  // loads in flight and waits for one block while the next is still arriving.
  auto load = [&](FragT (&kf)[2][KS], FragT (&vf)[2][KS], int j0) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int j = min(j0 + 16 * hh + r16, t1 - 1);
      const T* kr = j == old_len ? kn : kc + (size_t)j * D;
      const T* vr = j == old_len ? vn : vc + (size_t)j * D;
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

  // the G queries (rows past G zero) go to LDS as the A fragments of the logits, and
  // v_bar = s_v / n_e next to them; their reads are issued before the summary's
  constexpr int QPR = D * (int)sizeof(T) / 16;          // 16-byte pieces per query row
  constexpr int QPT = (16 * QPR + kEvThreads - 1) / kEvThreads;
  uint4 qv[QPT];
  const T* qh = reinterpret_cast<const T*>(e.q) + (size_t)head * G * D;
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int p = threadIdx.x + kEvThreads * u, row = p / QPR;
    qv[u] = (p < 16 * QPR && row < G)
                ? *reinterpret_cast<const uint4*>(qh + (size_t)row * D + (p % QPR) * (16 / (int)sizeof(T)))
                : make_uint4(0, 0, 0, 0);
  }
  const int ne = e.n_e[head];
  const float svv = threadIdx.x < D ? e.s_v[(size_t)head * D + threadIdx.x] : 0.f;

  build_summary<T, D>(e, head, sm);

#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int p = threadIdx.x + kEvThreads * u;
    if (p < 16 * QPR)
      *reinterpret_cast<uint4*>(&s_q[(p / QPR) * QRS + (p % QPR) * (16 / (int)sizeof(T))]) = qv[u];
  }
  const float cf = ne > 0 ? e.scale / (float)ne : 0.f;
  if (threadIdx.x < D) s_vbar[threadIdx.x] = ne > 0 ? svv / (float)ne : 0.f;
  auto process = [&](const FragT (&kf)[2][KS], const FragT (&vf)[2][KS], int j0) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      f32x4 lg = zero4();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) mma(lg, lds_frag(&s_q[r16 * QRS + 32 * ks + 8 * q4]), kf[hh][ks]);
      // every lane stores (no per-lane branch around a store): rows past t1 land in the
      // padding of the record planes, padded query slots in plane G + 1
      const int j = j0 + 16 * hh + r16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int g = 4 * q4 + i;
        rec[(size_t)(g < G ? g : G + 1) * ML + j] = lg[i] * c2;
      }
    }
    // S_tilde k: tile t = 2c + s holds dims 32c + 8 (lane/16) + 4s + i in lane rows
    // 4 (lane/16) + i, i.e. element 4s + i of the lane's V fragment c.
    float rr[2] = {0.f, 0.f};
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int c = t >> 1, s = t & 1;
      const int row = 32 * c + 8 * (r16 >> 2) + 4 * s + (r16 & 3);
      f32x4 ta[2] = {zero4(), zero4()};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if constexpr (sizeof(T) == 2) {
          const int col = scol<T>(row, 32 * ks + 8 * q4);
          const bf16x8 ah = lds_frag(&sm.hi[row * RS + col]);
          const bf16x8 al = lds_frag(&sm.lo[row * RS + col]);
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            mma(ta[hh], ah, kf[hh][ks]);
            mma(ta[hh], al, kf[hh][ks]);
          }
        } else {
          const f32x8 af = lds_frag(&sm.st[row * RS + 32 * ks + 8 * q4]);
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) mma(ta[hh], af, kf[hh][ks]);
        }
      }
      const float4 vb = *reinterpret_cast<const float4*>(&s_vbar[32 * c + 8 * q4 + 4 * s]);
      const float vbv[4] = {vb.x, vb.y, vb.z, vb.w};
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float r = elem_f(vf[hh][c], 4 * s + i) - vbv[i] - cf * ta[hh][i];
          rr[hh] += r * r;
        }
      // one tile's LDS reads in flight at a time: hoisting all of them would not fit
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      rr[hh] = cross_row_sum(rr[hh]);
      const int j = j0 + 16 * hh + r16;
      rec[(size_t)G * ML + j] = 0.5f * log2f(rr[hh]);  // the same value from four lanes
    }
  };
  __syncthreads();  // S_tilde and v_bar are in LDS

  // 32-row blocks j0, j0 + 128, ... of this wave; the next block's rows are requested
  // before the current block is processed (two register sets)
  for (; j0 < t1; j0 += 8 * kEvTB) {
    load(kb, vb, j0 + 4 * kEvTB);
    process(ka, va, j0);
    if (j0 + 4 * kEvTB >= t1) break;
    load(ka, va, j0 + 8 * kEvTB);
    process(kb, vb, j0 + 4 * kEvTB);
  }
  // The head's only workgroup selects right away: its records (and the appended row) are
  // visible to all of its waves after the barrier; no second launch.
  if (e.nslice == 1) {
    __syncthreads();
    select_head<T, D, GM, kEvThreads>(e, head, old_len, sel);
  }
}

// Selection as its own launch, one 512-thread workgroup per KV head (two fit on a CU, so
// a grid of a few hundred heads runs in one round): used when the scoring ran over
// several workgroups per head.
constexpr int kSelThreads = 512;

template <class T, int D, int GM>
__global__ void __launch_bounds__(kSelThreads) k_evict_select(EvictArgs e) {
  __shared__ SelLds<GM, kSelThreads / kWave, D> sl;
  select_head<T, D, GM, kSelThreads>(e, blockIdx.x, e.lens[blockIdx.x], sl);
}

template <class T, int D, int GM>
static hipError_t launch_evict_g(const EvictArgs& e, hipStream_t st) {
  hipLaunchKernelGGL((k_evict_scores<T, D, GM>), dim3(e.n_heads * e.nslice), dim3(kEvThreads), 0, st, e);
  if (e.nslice > 1)
    hipLaunchKernelGGL((k_evict_select<T, D, GM>), dim3(e.n_heads), dim3(kSelThreads), 0, st, e);
  return hipGetLastError();
}

template <class T, int D>
static hipError_t launch_evict_t(const EvictArgs& e, hipStream_t st) {
  if (e.G <= 4) return launch_evict_g<T, D, 4>(e, st);
  if (e.G <= 8) return launch_evict_g<T, D, 8>(e, st);
  return launch_evict_g<T, D, 16>(e, st);
}

hipError_t launch_evict(const EvictArgs& e, bool bf16, int d, hipStream_t st) {
  if (bf16) return d == 64 ? launch_evict_t<bf16_t, 64>(e, st) : launch_evict_t<bf16_t, 128>(e, st);
  return d == 64 ? launch_evict_t<float, 64>(e, st) : launch_evict_t<float, 128>(e, st);
}

}  // namespace mkv
