// Channel padding for head dimensions below the kernels' 32-channel minimum.
// A 16-channel q, k or v is copied into a 32-channel buffer whose extra
// channels are zero (zero key channels leave A_t, B_t, the states and the
// readout unchanged; zero value channels give zero outputs, which the
// readout's RMSNorm leaves out by averaging over the true d_v; the readout
// stores only the true channels).  Rows are 16-byte multiples.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

// dst[r][0..dst_bytes) = src[r][0..src_bytes) followed by zeros, in 16-byte
// pieces (dst_bytes >= src_bytes, both multiples of 16).
__global__ __launch_bounds__(kThreads)
void pad_rows_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, long long rows,
                     int src_chunks, int dst_chunks) {
  const long long total = rows * dst_chunks;
  for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < total;
       i += (long long)gridDim.x * kThreads) {
    const long long r = i / dst_chunks;
    const int c = (int)(i - r * dst_chunks);
    dst[i] = c < src_chunks ? src[r * src_chunks + c] : make_uint4(0u, 0u, 0u, 0u);
  }
}

unsigned copy_grid(long long chunks) {
  long long g = (chunks + kThreads - 1) / kThreads;
  if (g > 8192) g = 8192;
  return (unsigned)(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_pad_rows(const void* src, void* dst, long long rows, int src_bytes,
                           int dst_bytes, hipStream_t stream) {
  const int sc = src_bytes / 16, dc = dst_bytes / 16;
  hipLaunchKernelGGL(pad_rows_kernel, dim3(copy_grid(rows * dc)), dim3(kThreads), 0, stream,
                     static_cast<const uint4*>(src), static_cast<uint4*>(dst), rows, sc, dc);
  return hipGetLastError();
}

}  // namespace vda
