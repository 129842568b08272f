// probe.hip -- streaming-read probe (instrumentation): the rate at which a
// plain read of HBM proceeds on this device in the decode kernel's launch
// shape, for the roofline fraction of the attention kernels to be read
// against, and for the cost of the matrix-core operand load pattern.
//
// Two 256-thread workgroups per CU; workgroup g streams its own contiguous
// region of the buffer, its four waves taking 4 KB pieces (16 rows of 256
// bytes) round-robin with four non-temporal 16-byte loads per lane each:
//   lines:   load i covers rows 4i .. 4i+3 of the piece (lane = row lane/16,
//            chunk lane%16): whole 128-byte lines;
//   operand: load i covers bytes 64i .. 64i+63 of all 16 rows (lane = row
//            lane%16, chunk 4i + lane/16): the A-operand layout of a 16x16x32
//            matrix instruction, half of each line per load.
// Each wave XORs the words it read and stores one 16-byte value, so the
// loads are kept and the region each wave covered can be checked.
#include "mfma_util.h"
#include "uc_common.h"

namespace uc {
namespace {

using namespace mf;

template <int PATTERN>
__global__ __launch_bounds__(256, 2) void read_probe_kernel(const u4* __restrict__ buf,
                                                            uint64_t pieces_per_wg,
                                                            u4* __restrict__ sink) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const u4* region = buf + (uint64_t)blockIdx.x * pieces_per_wg * 256;
  const int off = PATTERN == 0 ? lane : (lane & 15) * 16 + (lane >> 4);
  const int step = PATTERN == 0 ? 64 : 4;
  u4 acc = u4{0, 0, 0, 0};
  for (uint64_t p = wave; p < pieces_per_wg; p += 4) {
    const u4* piece = region + p * 256 + off;
    u4 v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __builtin_nontemporal_load(piece + i * step);
    acc ^= (v[0] ^ v[1]) ^ (v[2] ^ v[3]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] ^= (uint32_t)__shfl_xor((int)acc[j], o, 64);
  }
  if (lane == 0) sink[blockIdx.x * 4 + wave] = acc;
}

}  // namespace

int read_probe_wgs() { return 2 * device_cus(); }

hipError_t launch_read_probe(const void* buf, size_t bytes, int pattern, void* sink,
                             hipStream_t st) {
  const int n = read_probe_wgs();
  const uint64_t pieces = bytes / 4096 / n;
  if (pattern == 0)
    hipLaunchKernelGGL(read_probe_kernel<0>, dim3(n), dim3(256), 0, st, (const u4*)buf, pieces,
                       (u4*)sink);
  else
    hipLaunchKernelGGL(read_probe_kernel<1>, dim3(n), dim3(256), 0, st, (const u4*)buf, pieces,
                       (u4*)sink);
  return hipGetLastError();
}

}  // namespace uc
