// Measurement kernels (laep_calib.h): a streaming copy, a blocked read and a
// bf16 MFMA loop.
#include "common.hpp"
#include "internal.hpp"

namespace laep {
namespace {

// Two 16-byte streaming loads in flight per thread before the streaming
// stores; launched with up to 64 Ki workgroups (the fastest of the variants
// measured: loads in flight 2-16, 2 Ki-256 Ki workgroups, ordinary or
// non-temporal accesses).
constexpr int kCopyUnroll = 2;
__global__ __launch_bounds__(256) void copy_kernel(const u32x4_t* __restrict__ src,
                                                   u32x4_t* __restrict__ dst, size_t n) {
  const size_t stride = (size_t)gridDim.x * blockDim.x * kCopyUnroll;
  for (size_t base = (size_t)blockIdx.x * blockDim.x * kCopyUnroll + threadIdx.x; base < n;
       base += stride) {
    u32x4_t v[kCopyUnroll];
#pragma unroll
    for (int j = 0; j < kCopyUnroll; ++j) {
      const size_t i = base + (size_t)j * blockDim.x;
      if (i < n) v[j] = ld_stream(src + i);
    }
#pragma unroll
    for (int j = 0; j < kCopyUnroll; ++j) {
      const size_t i = base + (size_t)j * blockDim.x;
      if (i < n) st_stream(dst + i, v[j]);
    }
  }
}

// Each workgroup reads its contiguous block: thread t its 16-byte chunks
// t, t + 512, ... (every load coalesced), all of them in flight at once, then
// writes the XOR of what it read (so the loads are not removed).
constexpr int kReadThreads = 512;
constexpr int kReadMaxChunks = 16;  // chunks per thread: blocks of up to 128 KB
__global__ __launch_bounds__(kReadThreads) void read_kernel(const u32x4_t* __restrict__ src,
                                                            int chunks, float* __restrict__ out) {
  const u32x4_t* p = src + (size_t)blockIdx.x * chunks * kReadThreads + threadIdx.x;
  u32x4_t v[kReadMaxChunks];
#pragma unroll
  for (int u = 0; u < kReadMaxChunks; ++u)
    if (u < chunks) v[u] = p[(size_t)u * kReadThreads];
  uint32_t x = 0;
#pragma unroll
  for (int u = 0; u < kReadMaxChunks; ++u)
    if (u < chunks) x ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  out[(size_t)blockIdx.x * kReadThreads + threadIdx.x] = __uint_as_float(x);
}

__global__ __launch_bounds__(512) void mfma_loop_kernel(int iters, float* __restrict__ out) {
  f32x16_t a0 = {}, a1 = {}, a2 = {}, a3 = {};
  bf16x8_t x, y;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    x[i] = (__bf16)(0.001f * (lane + i));
    y[i] = (__bf16)(0.002f * (i + 1));
  }
  for (int it = 0; it < iters; ++it) {
    a0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, a0, 0, 0, 0);
    a1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, a1, 0, 0, 0);
    a2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, a2, 0, 0, 0);
    a3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, a3, 0, 0, 0);
    a0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, a0, 0, 0, 0);
    a1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, a1, 0, 0, 0);
    a2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, a2, 0, 0, 0);
    a3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, a3, 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int r = 0; r < 16; ++r) s += a0[r] + a1[r] + a2[r] + a3[r];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace

hipError_t launch_calib_copy(const void* src, void* dst, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  const size_t n = bytes / 16;
  const size_t per_block = 256 * kCopyUnroll;
  const size_t blocks = (n + per_block - 1) / per_block;
  hipLaunchKernelGGL(copy_kernel, dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0,
                     s, static_cast<const u32x4_t*>(src), static_cast<u32x4_t*>(dst), n);
  return hipGetLastError();
}

hipError_t launch_calib_read(const void* src, size_t bytes, int block_bytes, float* out,
                             hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  const int chunks = block_bytes / (16 * kReadThreads);
  hipLaunchKernelGGL(read_kernel, dim3((unsigned)(bytes / block_bytes)), dim3(kReadThreads), 0, s,
                     static_cast<const u32x4_t*>(src), chunks, out);
  return hipGetLastError();
}

hipError_t launch_calib_mfma(int n_workgroups, int iters, float* out, hipStream_t s) {
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(n_workgroups), dim3(512), 0, s, iters, out);
  return hipGetLastError();
}

}  // namespace laep
