// js.hpp -- launcher of the Jensen--Shannon functional distance kernels
// (Sec. 4.4, JS distance; Appendix D.2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fgd {

// Device workspace bytes of one JS distance call (both dtypes' layouts).
int64_t js_workspace_bytes(int32_t bf16, int32_t M, int64_t U);

// Launches the row kernel, the per-token kernel and, when mean_out is given,
// the per-worker mean on `stream`; `workspace` holds js_workspace_bytes
// bytes (16-byte aligned) and num_cus sizes the row kernel's persistent
// grid.  False if a launch failed.
bool js_launch(const void *avg, const void *workers, int32_t bf16, int32_t M, int64_t U, int64_t K, int64_t ldk,
               int32_t k, double *d_out, double *mean_out, int32_t *topk_out, void *workspace, int num_cus,
               hipStream_t stream);

// Launches the row kernel's access pattern without its arithmetic on
// `stream` (see js_rows_pattern_kernel); it writes only the workspace's
// log-sum-exp parts.  False if the launch failed.
bool js_pattern_launch(const void *avg, const void *workers, int32_t bf16, int32_t M, int64_t U, int64_t K,
                       int64_t ldk, void *workspace, int num_cus, hipStream_t stream);

}  // namespace fgd
