// topk.hip - exact top-k per landmark row over stored score rows (Eq. top-k):
// one workgroup per row, or a fixed grid over a list of rows. The algorithm
// is in topk_row.hpp.
#include "kernels.hpp"
#include "topk_row.hpp"

namespace mita {

// One workgroup per row; with a row list, a fixed grid walks the *nrows
// listed rows (every workgroup exits at once when there are none).
template <int CAP, bool VEC, int ROWCAP>
__global__ __launch_bounds__(NT) void topk_kernel(const float *__restrict__ S, int32_t *__restrict__ idx, int N, int k,
                                                  const uint32_t *__restrict__ nrows,
                                                  const int32_t *__restrict__ rows) {
  __shared__ TopkSmem<CAP> sh;
  __shared__ __align__(16) float lrow[ROWCAP > 0 ? ROWCAP : 1];
  if (!rows) {
    const int64_t row = blockIdx.x;
    topk_row<CAP, VEC, ROWCAP>(sh, lrow, S + row * (int64_t)N, idx + row * (int64_t)k, N, k);
    return;
  }
  topk_listed_body<CAP, VEC, ROWCAP>(sh, lrow, (int)blockIdx.x, (int)gridDim.x, S, idx, N, k, nrows, rows);
}

template <int CAP, int ROWCAP>
static hipError_t topk_t(const mita_cfg_t &c, const float *S, int32_t *idx, hipStream_t st, const uint32_t *nrows,
                         const int32_t *rows) {
  const int64_t all = BH(c) * c.M;
  const unsigned grid = (unsigned)(rows ? (all < 512 ? all : 512) : all);
  if (c.N % 4 == 0)
    hipLaunchKernelGGL((topk_kernel<CAP, true, ROWCAP>), dim3(grid), dim3(NT), 0, st, S, idx, c.N, c.k, nrows, rows);
  else
    hipLaunchKernelGGL((topk_kernel<CAP, false, ROWCAP>), dim3(grid), dim3(NT), 0, st, S, idx, c.N, c.k, nrows, rows);
  return launched("topk_kernel", st);
}

// Rows up to 16384 scores (64 KiB) are copied into LDS once; longer rows are
// streamed from memory in every pass.
hipError_t launch_topk(const mita_cfg_t &c, const float *S, int32_t *idx, hipStream_t st, const uint32_t *nrows,
                       const int32_t *rows) {
  if (c.N <= 4096) return topk_t<512, 4096>(c, S, idx, st, nrows, rows);
  if (c.N <= 16384) return topk_t<512, 16384>(c, S, idx, st, nrows, rows);
  return topk_t<2048, 0>(c, S, idx, st, nrows, rows);
}

}  // namespace mita
