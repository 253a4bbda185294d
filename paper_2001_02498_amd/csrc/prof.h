// Launch timing scopes (see prof.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "common.h"

namespace gcn {

enum Kind : int {
    K_PAIR_SUMS = 0,
    K_LIST_SUMS,
    K_GEMM_FWD,
    K_GEMM_CLS,
    K_GEMM_DX,
    K_GEMM_CLS_DX,
    K_GEMM_DW,
    K_GEMM_CLS_DW,
    K_SGD,
    K_LOSS_ROWS,
    K_LOSS_MEAN,
    K_SPLITK_FINISH,
    // the GEMM roles again, bf16 operands
    K_GEMM_FWD_BF16,
    K_GEMM_CLS_BF16,
    K_GEMM_DX_BF16,
    K_GEMM_CLS_DX_BF16,
    K_GEMM_DW_BF16,
    K_GEMM_CLS_DW_BF16,
    K_TO_BF16,
    // the first layer's products (K or M = f_in), fp32 and bf16 operands
    K_GEMM_FWD_IN,
    K_GEMM_DW_IN,
    K_GEMM_FWD_IN_BF16,
    K_GEMM_DW_IN_BF16,
    // rows of the full graph's features and labels for a sampled minibatch
    K_GATHER,
    // streaming read of a buffer larger than the caches (measurement)
    K_READ_PROBE,
    K_COUNT
};

const char* kind_name(int k);

// Records an event pair around the launches made during its lifetime when
// timing is enabled; a no-op otherwise.
class ProfScope {
   public:
    ProfScope(hipStream_t s, int kind, double flops, double bytes);
    ~ProfScope();
    ProfScope(const ProfScope&) = delete;
    ProfScope& operator=(const ProfScope&) = delete;

   private:
    hipStream_t s_;
    int64_t idx_;
};

}  // namespace gcn
