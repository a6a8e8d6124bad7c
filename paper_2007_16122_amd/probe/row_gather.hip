// row_gather.hip -- the plainest gather of 32-byte rows (libcold_probe.so):
// a measurement aid that times scattered row reads on their own, beside the
// scoring library.  Thread j copies 16-byte half j % 2 of row j / 2: the two
// threads of a row read its index together and its two halves side by side,
// consecutive threads write consecutive 16 bytes, so index reads and stores
// are coalesced and only the table reads scatter.  Of the simple forms
// timed on the serving workload's rows (one row or 2, 4, 8, 16 rows per
// thread, a quarter row per thread, workgroups of 64 to 1,024 threads) this
// one was the fastest.
#include <hip/hip_runtime.h>

#include "cold_probe.h"

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void row_gather_probe_kernel(const uint4 *__restrict__ table,
                                                                   int64_t table_rows,
                                                                   const int64_t *__restrict__ idx,
                                                                   uint4 *__restrict__ out, int64_t n) {
  const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t i = j >> 1;
  if (i >= n) return;
  const int64_t r = idx[i];
  const int64_t row = r >= 0 && r < table_rows ? r : 0;
  out[j] = table[2 * row + (j & 1)];
}

}  // namespace

extern "C" int cold_probe_row_gather(const void *table, int64_t table_rows, const int64_t *idx,
                                     void *out, int64_t n, void *stream) {
  if (!table || !idx || !out || n < 0 || table_rows <= 0) return -1;
  if (n == 0) return 0;
  const int64_t blocks = (2 * n + kThreads - 1) / kThreads;
  if (n > (INT64_MAX >> 2) || blocks > 0x7FFFFFFF) return -1;
  hipLaunchKernelGGL(row_gather_probe_kernel, dim3((unsigned)blocks), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint4 *>(table), table_rows,
                     idx, static_cast<uint4 *>(out), n);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
