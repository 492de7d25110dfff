// Launch context: either enqueues kernels on a stream, or (dry run) only
// records how much split-K workspace the same sequence of GEMMs needs, so the
// size queries and the real calls can never disagree.
#pragma once

#include "gemm.hpp"

namespace pf {

struct Runner {
  bool dry;
  hipStream_t stream;
  float* gemm_ws;      // split-K partials (may be NULL in a dry run)
  size_t gemm_need;    // dry run: max bytes any GEMM asked for
  hipError_t err;

  explicit Runner(bool dry_run, hipStream_t s = nullptr, float* ws = nullptr)
      : dry(dry_run), stream(s), gemm_ws(ws), gemm_need(0), err(hipSuccess) {}

  bool ok() const { return err == hipSuccess; }

  template <typename T, int LA, int LB, class Epi>
  void gemm(const GemmProblem& pr, const Epi& epi) {
    if (!ok()) return;
    if (dry) {
      const size_t need = gemm_workspace_bytes<T>(pr, kPlanCUsGemm);
      if (need > gemm_need) gemm_need = need;
      return;
    }
    err = run_gemm<T, LA, LB>(pr, epi, gemm_ws, kPlanCUsGemm, stream);
  }

  template <class F>
  void launch(F&& f) {
    if (!ok() || dry) return;
    err = f();
  }

  static constexpr int kPlanCUsGemm = 256;
};

// Zero-fill of a device byte range with a kernel (no memset nodes, so the
// sequence stays valid inside a captured HIP graph).
hipError_t fill_zero(void* p, size_t bytes, hipStream_t stream);

}  // namespace pf
