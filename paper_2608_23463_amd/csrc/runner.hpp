// Launch context: either enqueues kernels on a stream, or (dry run) only
// records how much split-K workspace the same sequence of GEMMs needs, so the
// size queries and the real calls can never disagree.
#pragma once

#include "gemm.hpp"
#include "trace.hpp"

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

  // C = A B^T through `epi`, with a deterministic split-K through gemm_ws when
  // the plan asks for it. `label` names the launch for tracing.
  template <typename T, int LA, int LB, class Epi>
  void gemm(const char* label, const GemmProblem& pr, const Epi& epi) {
    if (!ok() || pr.M <= 0 || pr.N <= 0) return;
    GemmPlan pl = plan_gemm<T>(pr, kPlanCUsGemm);
    if (dry) {
      if (pl.splits > 1) {
        const size_t need = (size_t)pl.splits * pr.M * pr.N * sizeof(float);
        if (need > gemm_need) gemm_need = need;
      }
      return;
    }
    if (pl.splits <= 1 || gemm_ws == nullptr) {
      pl.splits = 1;
      pl.k_slice = std::max(pl.bk, ((pr.K + pl.bk - 1) / pl.bk) * pl.bk);
      timed(label, [&] { return launch_gemm_plan<T, LA, LB>(pr, pl, epi, stream); });
      return;
    }
    EpiPartial part{gemm_ws, pr.N, (int64_t)pr.M * pr.N};
    timed(label, [&] { return launch_gemm_plan<T, LA, LB>(pr, pl, part, stream); });
    if (!ok()) return;
    const int64_t total = (int64_t)pr.M * pr.N;
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
    timed("splitk_reduce", [&] {
      hipLaunchKernelGGL((splitk_reduce_kernel<Epi>), dim3(blocks), dim3(256), 0, stream, gemm_ws, pl.splits, pr.M,
                         pr.N, epi);
      return hipGetLastError();
    });
  }

  template <class F>
  void launch(const char* label, F&& f) {
    if (!ok() || dry) return;
    timed(label, f);
  }

  template <class F>
  void timed(const char* label, F&& f) {
    const bool tr = trace_on();
    if (tr) trace_begin(label, stream);
    err = f();
    if (tr) trace_end(stream);
  }

  static constexpr int kPlanCUsGemm = 256;
};

// Zero-fill of a device byte range with a kernel (no memset nodes, so the
// sequence stays valid inside a captured HIP graph).
hipError_t fill_zero(void* p, size_t bytes, hipStream_t stream);

}  // namespace pf
