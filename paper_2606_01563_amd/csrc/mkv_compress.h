// Host <-> device interface of the compress kernels (compress.hip): the argument block
// passed by value and the launcher the C ABI layer calls.  Pointers are device pointers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mkv {

// Most 64-token tiles one workgroup of the window-row/covariance, window-mass and
// residual passes takes: its per-token results wait in LDS until its tile loop ends.
constexpr int kRowsMaxTiles = 64;
constexpr int kMassMaxTiles = 8;
constexpr int kResMaxTiles = 32;

struct CompressArgs {
  const void* q_win;        // [B, Hq, w, D]
  const void* k;            // [B, Hkv, N, D]
  const void* v;
  void* k_out;              // [B, Hkv, cap, D]
  void* v_out;
  int32_t* idx_out;         // [B, Hkv, L']
  int32_t* lens_out;        // [B, Hkv]
  int32_t* n_e;             // [B, Hkv]
  float* s_k;               // [B, Hkv, D]
  float* s_v;
  void* S;                  // [B, Hkv, D, D] fp32, or bf16 when S_bf16
  int S_bf16;               // the output S in bf16 (RNE of the fp32 sum)
  // workspace
  float* rowpart;           // [H, nsl1, R, 2]   per-slice (max log2, sum) of each window row
  float* rowstat;           // [H, R, 2]         (max log2, 1/Z)
  float* vnorm;             // [H, n_c]          ||v_j||
  float* abar;              // [H, n_c]          pooled window mass
  float* score0;            // [H, n_c]          provisional score
  float* score;             // [H, n_c]          moment-round score
  int32_t* kept0;           // [H, kmax]         provisional kept positions (ascending)
  int32_t* kept;            // [H, kmax]         final kept positions (ascending)
  uint32_t* tk_hh;          // [2, H, 2048]      top-k: per-head histograms of key bits 30..20
                            //                   of the first and the final scores
  int32_t* tk_state;        // [H, 2]            top-k: bin of the k-th key, count above it
  int32_t* tk_cnt;          // [H, ntk, 2]       top-k: per slice, keys above the bin, in it
  uint32_t* tk_cand;        // [H, ntk, 2048]    top-k: per slice, the keys in the bin
  float* spart;             // [H, nslot, D, D]  covariance partials (after the row-statistics
                            // launch, slot 0 holds the sum of slots 0 .. nsl1 - 1)
  float* svkpart;           // [H, nslot, 2, D]  (s_v, s_k) partials
  float* s0;                // [H, D, D]         raw S of the provisional evicted set
  float* sv0;               // [H, D]            its s_v
  float* sk0;               // [H, D]            its s_k
  int B, Hq, Hkv, G, N, L, w, n_s, chunk, mi_rounds, cap, D;
  int H;                    // B * Hkv
  int R;                    // G * w window rows per KV head
  int n_c;                  // N - w - n_s candidates
  int k_keep;               // L - n_s - w
  int kmax;                 // row capacity of kept/gath buffers (>= k_keep, >= 1)
  int ntile;                // ceil(N / 64)
  int nsl1, tps1;           // window-row/covariance pass: slices, tiles per slice
                            // (tps1 <= kRowsMaxTiles)
  int nsl2, tps2;           // window-mass pass: slices, tiles per slice (<= kMassMaxTiles)
  int nslot;                // nsl1 + ntk: the candidate slices' slots, then one slot per
                            // top-k slice for the covariance of its kept rows (subtracted)
                            // or, when a head's evicted rows are the fewer, its evicted rows'

  int nsl3, tps3;           // residual pass: slices over candidate tiles of 64 (<= kResMaxTiles)
  int ntk;                  // top-k slices of 2048 candidates
  // head-adaptive budgets (adaptive = 1): a per-sequence selection over the layer
  int adaptive;
  int32_t* kh;              // [H] candidates kept per head, or null (k_keep everywhere)
  int32_t* kept_all;        // [B, Hkv*k_keep] layer-wide kept candidates (head*n_c + j)
  uint32_t* tk_hs;          // [B, 2048] key histogram of abar over the layer
  int32_t* tk_state_g;      // [B, 2], and the candidate buffers of that selection:
  int32_t* tk_cnt_g;        // [B, ntk_g, 2]
  uint32_t* tk_cand_g;      // [B, ntk_g, 2048]
  int ntk_g;                // slices of the layer-wide selection
  int idx_stride;           // entries per head of idx_out
  float scale, tau;
};

// Full compress pipeline on one stream (see compress.hip for the stage list).
hipError_t launch_compress(const CompressArgs& a, bool bf16, hipStream_t st,
                           float* dbg_abar, float* dbg_score0, float* dbg_score,
                           int32_t* dbg_kept0);

}  // namespace mkv
