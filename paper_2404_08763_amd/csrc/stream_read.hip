// Attainable read bandwidth: a plain stream over a device buffer with the
// weight kernels' own load (16 bytes per lane, non-temporal, through a
// buffer resource), so the weight-streaming kernels can be rated against
// what this device actually delivers as well as against its rated peak.
// Nothing of the method is computed here.
#include "device.hpp"
#include "internal.hpp"

namespace cats {

static_assert(kStreamReadMaxBytes <= kBufMaxBytes, "one buffer resource covers the stream");
constexpr int kStreamThreads = 256;
constexpr int kStreamWaves = kStreamThreads / kWaveSize;
constexpr uint32_t kStreamUnit = kWaveSize * 16;  // one wave load: 1 KB

// U loads of 1 KB per wave in flight per step.  RUNS = false: load u of
// step s, wave w covers unit (s U + u) NW + w (the waves of the grid side by
// side); RUNS = true: unit (s NW + w) U + u (each wave a run of U KB).  The
// xor of the words feeds a store that practically never happens, so no
// load can be dropped and nothing is written.
template <int U, bool RUNS>
__global__ __launch_bounds__(kStreamThreads) void k_stream_read(const void* buf, uint32_t bytes, uint32_t* sink) {
  const int lane = threadIdx.x & (kWaveSize - 1);
  const uint32_t nw = gridDim.x * kStreamWaves;
  const uint32_t w = blockIdx.x * kStreamWaves + threadIdx.x / kWaveSize;
  const uint32_t units = (bytes + kStreamUnit - 1) / kStreamUnit;
  const uint32_t steps = (units + nw * U - 1) / (nw * U);
  const __amdgpu_buffer_rsrc_t r = make_rsrc(buf, bytes);
  uint32_t acc = 0;
  for (uint32_t s = 0; s < steps; ++s) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t unit = RUNS ? (s * nw + w) * U + u : (s * U + u) * nw + w;
      v[u] = ld_buf16_stream(r, unit < units ? unit * kStreamUnit + (uint32_t)lane * 16u : kOOB);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (acc == 0x9e3779b9u) sink[blockIdx.x] = acc;
}

template <int U>
static hipError_t launch_stream_u(bool runs, const void* buf, uint32_t bytes, int blocks, uint32_t* sink,
                                  hipStream_t s) {
  KernelTimer timer("stream_read", s);
  if (runs)
    hipExtLaunchKernelGGL((k_stream_read<U, true>), dim3(blocks), dim3(kStreamThreads), 0, s, timer.start(),
                          timer.stop(), 0, buf, bytes, sink);
  else
    hipExtLaunchKernelGGL((k_stream_read<U, false>), dim3(blocks), dim3(kStreamThreads), 0, s, timer.start(),
                          timer.stop(), 0, buf, bytes, sink);
  return hipGetLastError();
}

hipError_t launch_stream_read(const void* buf, uint32_t bytes, int blocks, int inflight, bool runs, uint32_t* sink,
                              hipStream_t s) {
  switch (inflight) {
    case 4: return launch_stream_u<4>(runs, buf, bytes, blocks, sink, s);
    case 8: return launch_stream_u<8>(runs, buf, bytes, blocks, sink, s);
    case 16: return launch_stream_u<16>(runs, buf, bytes, blocks, sink, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace cats
