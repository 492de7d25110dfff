// Fused level-1 decompression + gated injection (Eq. 10 with Eq. 12), bf16.
#pragma once

#include "common.hpp"

namespace pf {

// Rows r of S (the level-1 decompression input, [M, Ks]) and of X viewed as
// [M, k N] (row stride lda_x = k N); position p < k selects column block
// p N of X, rows p N .. of the level-1 decompression weight W_d [k N, Ks]
// and of C = [W_gd W_d[p]]_p [k N, Ks]. W_g [N, 2 N] (first N columns used,
// row stride ldb_g); bias_g: b' [k, N] fp32 (b_g + W_gd b_d[p]); bias_d:
// b_d [k N] or NULL. Y (and, when not NULL, the saved Delta and G) share
// X's layout.
struct FusedGateParams {
  const bf16* s;
  const bf16* x;
  const bf16* wc;
  const bf16* wd;
  const bf16* wg;
  const float* bias_g;
  const bf16* bias_d;
  bf16* y;
  bf16* delta_out;
  bf16* g_out;
  int M;          // rows (batch * level-1 groups)
  int k;          // positions per group (k_1)
  int64_t N;      // d_fine
  int64_t Ks;     // d_1 (the decompression input width)
  int64_t lda_s, lda_x, ldb_g;
  int tiles_m, tiles_n;  // set by the launcher
};

// The kernel takes whole 128-channel tiles and 64-wide K steps, over a level-1
// input at least 128 wide.
bool fused_gate_supported(int64_t N, int64_t Ks);
hipError_t launch_fused_gate(const FusedGateParams& p, hipStream_t stream);

}  // namespace pf
