// Top-tau block selection kernels (paper Alg. 1 step 7 / Alg. 2 step 6;
// forced first and last blocks per Sec. 4.1): one 256-thread workgroup per
// row, each running the radix selection of select_row.h.
#include "select_row.h"
#include "sw_internal.h"

namespace sw {

template <int MAXE>
__global__ __launch_bounds__(256) void select_prefill_kernel(const double* __restrict__ R,
                                                             SeqMeta m, int k, int pct,
                                                             uint32_t flags,
                                                             int32_t* __restrict__ idx,
                                                             int32_t* __restrict__ cnt, int kmax) {
  const int row = blockIdx.x;
  const int s = seq_of_block(m, row);
  const int i = row - m.blk_start[s];
  const int b = m.blk_start[s + 1] - m.blk_start[s];
  const double* vals = R + m.mat_start[s] + (long long)i * b;
  const int first = (flags & SW_FORCE_FIRST) ? 0 : -1;
  const int last = (flags & SW_FORCE_LAST) ? i : -1;
  select_row_dev<MAXE>(vals, i + 1, first, last, k, pct, idx + (long long)row * kmax, cnt + row, kmax);
}

// One row per sequence (Alg. 2 step 6): the walk row over key blocks
// 0..b_cur of the token at pos[b]; forced set {0, b_cur}.
template <int MAXE>
__global__ __launch_bounds__(256) void select_decode_kernel(const double* __restrict__ rows,
                                                            int b_max, int B,
                                                            const int32_t* __restrict__ pos, int k,
                                                            int pct, uint32_t flags,
                                                            int32_t* __restrict__ idx,
                                                            int32_t* __restrict__ cnt, int kmax) {
  const int bi = blockIdx.x;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  const int first = (flags & SW_FORCE_FIRST) ? 0 : -1;
  const int last = (flags & SW_FORCE_LAST) ? bc : -1;
  select_row_dev<MAXE>(rows + (long long)bi * b_max, bc + 1, first, last, k, pct,
                 idx + (long long)bi * kmax, cnt + bi, kmax);
}

hipError_t launch_select_decode(const double* rows, int batch, int b_max, int B,
                                const int32_t* pos, int k, int pct, uint32_t flags, int32_t* idx,
                                int32_t* cnt, int kmax, hipStream_t st) {
#define SW_SEL_DEC(E)                                                                            \
  hipLaunchKernelGGL(select_decode_kernel<E>, dim3((unsigned)batch), dim3(256), 0, st, rows, b_max, \
                     B, pos, k, pct, flags, idx, cnt, kmax)
  switch (row_maxe(b_max)) {
    case 2: SW_SEL_DEC(2); break;
    case 4: SW_SEL_DEC(4); break;
    case 8: SW_SEL_DEC(8); break;
    default: SW_SEL_DEC(16); break;
  }
#undef SW_SEL_DEC
  return hipGetLastError();
}

hipError_t launch_select(const double* R, const SeqMeta& meta, int64_t nb, int k, int pct,
                         uint32_t flags, int32_t* idx, int32_t* cnt, int kmax, hipStream_t st) {
#define SW_SEL_PRE(E)                                                                         \
  hipLaunchKernelGGL(select_prefill_kernel<E>, dim3((unsigned)nb), dim3(256), 0, st, R, meta, k, \
                     pct, flags, idx, cnt, kmax)
  switch (row_maxe(meta.max_b)) {
    case 2: SW_SEL_PRE(2); break;
    case 4: SW_SEL_PRE(4); break;
    case 8: SW_SEL_PRE(8); break;
    default: SW_SEL_PRE(16); break;
  }
#undef SW_SEL_PRE
  return hipGetLastError();
}

}  // namespace sw
