// Launchers shared between the kernel translation units and the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sw_common.h"

namespace sw {

int64_t sketch_workspace_bytes(int h_q, int h_kv, int d, int64_t nb);

hipError_t launch_sketch(int dtype, const void* Q, const void* K, int h_q, int h_kv, int d,
                         const SeqMeta& meta, int64_t nb, long long N, const int8_t* signs,
                         const int32_t* cols, int r, double* Qs, double* Ks, double* A,
                         double* A_scale, double* Qbar, double* Kbar, void* ws, hipStream_t st);

hipError_t launch_walk(const double* A, const double* A_scale, int s_exp, const SeqMeta& meta,
                       int64_t nb, const double* R_prev, double* R_out, hipStream_t st);

hipError_t launch_select(const double* R, const SeqMeta& meta, int64_t nb, int k, int pct,
                         uint32_t flags, int32_t* idx, int32_t* cnt, int kmax, hipStream_t st);

hipError_t launch_attn_prefill(int dtype, const void* Q, const void* K, const void* V, int h_q,
                               int h_kv, int d, long long N, const SeqMeta& meta, int64_t nb,
                               const int32_t* idx, const int32_t* cnt, int kmax, float scale,
                               void* O, float* lse, hipStream_t st);

}  // namespace sw
