// Streaming-read ceiling: the HBM read rate a kernel reaches with the weight
// stream's access pattern (one 16-wave block per CU, 1 KB wavefront loads of
// streamed-once data, two batches of four loads per wave in flight), used to
// put the verify step's bandwidth beside a rate measured on the same device.
#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace specdec {

namespace {

constexpr int kStreamWaves = 16;
constexpr int kStreamBatch = 4;  // loads per wave per batch

// Block b reads the 1 KB chunks [b * per, min((b + 1) * per, n)) of buf; wave w
// takes chunks w, w + 16, ... of the block's range.  Every loaded word is
// XOR-ed into one value per lane, stored only if it equals a value no input
// here produces, so no load can be dropped and nothing is written in practice.
__global__ __launch_bounds__(64 * kStreamWaves) void stream_read_kernel(const unsigned char* buf, uint64_t n_chunks,
                                                                       uint64_t per, uint32_t* sink) {
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint64_t c0 = (uint64_t)blockIdx.x * per;
  if (c0 >= n_chunks) return;
  const uint32_t nc = (uint32_t)std::min<uint64_t>(per, n_chunks - c0);
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(buf + c0 * 1024), (short)0, nc * 1024u, 0x00020000);
  const uint32_t mine = nc > (uint32_t)wave ? (nc - wave + kStreamWaves - 1) / kStreamWaves : 0;
  const uint32_t nbat = (mine + kStreamBatch - 1) / kStreamBatch;
  auto load = [&](uint32_t bi, u32x4 (&v)[kStreamBatch]) {
#pragma unroll
    for (int u = 0; u < kStreamBatch; ++u) {
      const uint32_t i = bi * kStreamBatch + u;        // index in this wave's list
      const uint32_t c = (uint32_t)wave + i * kStreamWaves;
      v[u] = __builtin_amdgcn_raw_buffer_load_b128(r, (c * 1024u + lane * 16u) | ((uint32_t)(i >= mine) << 31), 0,
                                                   2 /* streamed once */);
    }
  };
  uint32_t acc = 0;
  u32x4 a[kStreamBatch], b[kStreamBatch];
  if (nbat > 0) load(0, a);
  if (nbat > 1) load(1, b);
  for (uint32_t bi = 0; bi < nbat; bi += 2) {
#pragma unroll
    for (int u = 0; u < kStreamBatch; ++u) acc ^= a[u][0] ^ a[u][3];
    if (bi + 2 < nbat) load(bi + 2, a);
    if (bi + 1 >= nbat) break;
#pragma unroll
    for (int u = 0; u < kStreamBatch; ++u) acc ^= b[u][0] ^ b[u][3];
    if (bi + 3 < nbat) load(bi + 3, b);
  }
  if (acc == 0x9E3779B9u) sink[0] = acc;
}

}  // namespace

hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, hipStream_t s) {
  const uint64_t n_chunks = bytes / 1024;
  if (n_chunks == 0) return hipSuccess;
  const int blocks = device_compute_units();
  const uint64_t per = (n_chunks + blocks - 1) / blocks;
  if (per * 1024 > 0xFFFFFFFFull) return hipErrorInvalidValue;  // (one block's range within a 32-bit offset)
  hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(64 * kStreamWaves), 0, s,
                     (const unsigned char*)buf, n_chunks, per, sink);
  return hipGetLastError();
}

}  // namespace specdec
