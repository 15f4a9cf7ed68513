// Streaming-read probe (measurement, not part of the decode path): the rate at which this
// GPU reads a span from HBM, by the decode attention's own access method and by plain
// register loads, so that the benchmark can set the attention's achieved bandwidth beside
// the ceiling it measures in the same run (gfx950).
//
//   method 0: WGs of 8 waves, one contiguous span per WG; each wave streams 16 KiB batches
//             (sixteen 16-byte direct global -> LDS loads per lane, non-temporal policy)
//             with one batch in flight, the next one issued as soon as the current one has
//             been read back from LDS: the decode kernel's K/V tile stream;
//   method 1: WGs of 512 threads striding over the buffer, eight 16-byte non-temporal
//             register loads in flight per thread.
// Every 32-bit word is read once; WG g writes the XOR of the words it read to sink[g] (the
// XOR over all WGs is the XOR of the buffer: a check that the probe read all of it).
#include "td_internal.h"

namespace td {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeWaves = 8;
constexpr int kProbeBatch = 16;             // 1 KiB loads per wave batch (16 KiB)
constexpr int kProbeRegThreads = 512;
constexpr int kProbeRegUnroll = 8;

__device__ inline unsigned wave_xor(unsigned v) {
  for (int o = 32; o > 0; o >>= 1) v ^= __shfl_xor(v, o);
  return v;
}

__device__ inline void block_xor_store(unsigned acc, unsigned* red, unsigned* sink) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  acc = wave_xor(acc);
  if (lane == 0) red[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned x = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) x ^= red[w];
    sink[blockIdx.x] = x;
  }
}

__global__ __launch_bounds__(kProbeWaves * 64) void k_read_lds(const u32x4* __restrict__ p, size_t n16,
                                                              unsigned* sink) {
  __shared__ u32x4 buf[kProbeWaves][kProbeBatch][64];
  __shared__ unsigned red[kProbeWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr size_t batch = (size_t)kProbeBatch * 64;  // 16-byte words per wave batch
  // this WG's span: whole batches of the WG's 8 waves, the last WG's cut at the end
  const size_t per = ((n16 + gridDim.x - 1) / gridDim.x + batch - 1) / batch * batch;
  const size_t b0 = min(n16, (size_t)blockIdx.x * per), b1 = min(n16, b0 + per);
  const long nb = (long)((b1 - b0 + batch - 1) / batch);  // batches of this WG
  const long mine = nb > wave ? (nb - wave + kProbeWaves - 1) / kProbeWaves : 0;
  auto issue = [&](long k) __attribute__((always_inline)) {
    const size_t base = b0 + (size_t)(wave + k * kProbeWaves) * batch;
#pragma unroll
    for (int u = 0; u < kProbeBatch; ++u) {
      const size_t i = min(base + (size_t)u * 64 + lane, b1 - 1);  // (the tail re-reads its last word)
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(p + i),
                                       (__attribute__((address_space(3))) void*)&buf[wave][u][0], 16, 0, 2);
    }
  };
  unsigned acc = 0;
  if (mine > 0) issue(0);
  for (long k = 0; k < mine; ++k) {
    __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8));  // vmcnt(0): the batch is in LDS
    const size_t base = b0 + (size_t)(wave + k * kProbeWaves) * batch;
    u32x4 v[kProbeBatch];
#pragma unroll
    for (int u = 0; u < kProbeBatch; ++u) v[u] = buf[wave][u][lane];
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8));  // lgkmcnt(0): read back
    if (k + 1 < mine) issue(k + 1);
#pragma unroll
    for (int u = 0; u < kProbeBatch; ++u)
      if (base + (size_t)u * 64 + lane < b1) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  block_xor_store(acc, red, sink);
}

__global__ __launch_bounds__(kProbeRegThreads) void k_read_reg(const u32x4* __restrict__ p, size_t n16,
                                                              unsigned* sink) {
  __shared__ unsigned red[kProbeRegThreads / 64];
  unsigned acc = 0;
  const size_t step = (size_t)gridDim.x * kProbeRegThreads * kProbeRegUnroll;
  for (size_t base = (size_t)blockIdx.x * kProbeRegThreads * kProbeRegUnroll; base < n16; base += step) {
    u32x4 v[kProbeRegUnroll];
#pragma unroll
    for (int u = 0; u < kProbeRegUnroll; ++u) {
      const size_t i = base + (size_t)u * kProbeRegThreads + threadIdx.x;
      v[u] = i < n16 ? __builtin_nontemporal_load(p + i) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < kProbeRegUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  block_xor_store(acc, red, sink);
}

}  // namespace

}  // namespace td

extern "C" td_status td_read_probe(const void* d_buf, size_t bytes, int32_t method, int32_t n_wgs,
                                   uint32_t* d_sink, hipEvent_t ev_start, hipEvent_t ev_stop,
                                   hipStream_t stream) {
  using namespace td;
  set_error_without_context("");
  if (!d_buf || !d_sink || (reinterpret_cast<uintptr_t>(d_buf) & 15u) != 0) {
    set_error_without_context("td_read_probe: buffer and sink are required, the buffer 16-byte aligned");
    return TD_EINVAL;
  }
  if (bytes == 0 || bytes % 16 != 0 || n_wgs < 1 || n_wgs > 65536 || (method != 0 && method != 1)) {
    set_error_without_context("td_read_probe: bytes a positive multiple of 16, n_wgs in [1, 65536], method 0 or 1");
    return TD_EINVAL;
  }
  const size_t n16 = bytes / 16;
  if (method == 0)
    hipExtLaunchKernelGGL(k_read_lds, dim3(n_wgs), dim3(kProbeWaves * 64), 0, stream, ev_start, ev_stop, 0,
                          static_cast<const u32x4*>(d_buf), n16, reinterpret_cast<unsigned*>(d_sink));
  else
    hipExtLaunchKernelGGL(k_read_reg, dim3(n_wgs), dim3(kProbeRegThreads), 0, stream, ev_start, ev_stop, 0,
                          static_cast<const u32x4*>(d_buf), n16, reinterpret_cast<unsigned*>(d_sink));
  if (hipGetLastError() != hipSuccess) {
    set_error_without_context("td_read_probe: launch failed");
    return TD_EHIP;
  }
  return TD_OK;
}
