// gfx950 probes (see include/ozaki2_probes.h): E4M3 encoding, FP32
// accumulation exactness of the FP8 MFMA, MFMA peak (near-constant and
// digit-plane operands), HBM copy peak.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstring>

#include "../../include/ozaki2.h"
#include "../../include/ozaki2_probes.h"

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

__global__ void k_e4m3(const float* __restrict__ x, uint8_t* __restrict__ out, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int w = __builtin_amdgcn_cvt_pk_fp8_f32(x[i], 0.0f, 0, false);
  out[i] = (uint8_t)(w & 0xFF);
}

__global__ void __launch_bounds__(64) k_accum(const uint8_t* __restrict__ a,
                                              const uint8_t* __restrict__ b, int chain,
                                              float* __restrict__ out) {
  const int l = threadIdx.x;
  v8i av, bv;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    av[i] = (int)(a[32 * l + 4 * i] | (a[32 * l + 4 * i + 1] << 8) | (a[32 * l + 4 * i + 2] << 16) |
                  ((uint32_t)a[32 * l + 4 * i + 3] << 24));
    bv[i] = (int)(b[32 * l + 4 * i] | (b[32 * l + 4 * i + 1] << 8) | (b[32 * l + 4 * i + 2] << 16) |
                  ((uint32_t)b[32 * l + 4 * i + 3] << 24));
  }
  v16f acc = v16f{0.f};
  for (int c = 0; c < chain; ++c)
    acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, acc, 0, 0, 0, 0, 0, 0);
#pragma unroll
  for (int e = 0; e < 16; ++e) out[16 * l + e] = acc[e];
}

// grid-stride 16-byte copy; 4 workgroups per CU measured fastest among
// 1K-64K workgroups and 1-8 loads in flight per lane
__global__ void __launch_bounds__(256) k_copy(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                              size_t n16) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    dst[i] = src[i];
}

// 8 independent accumulators per wave, 2 waves per SIMD (512 threads per CU)
__global__ void __launch_bounds__(512) k_mfma_peak(int iters, float* sink) {
  v8i a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = 0x38383838 + (int)threadIdx.x;
    b[i] = 0x30303030 + i;
  }
  v16f acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = v16f{0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc[j], 0, 0, 0, 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  if (s == 1.0e30f) sink[threadIdx.x] = s;   // keeps the MFMAs live; never true
}

// The residue GEMM's inner loop on its own data: 64 KiB of LDS holding E4M3
// bytes of digits drawn uniformly from [-11, 11] (the balanced base-23 digits
// of a square-modulus plane), and per K = 64 step a wave reads the next
// step's 4 + 2 fragments (12 x 16 B per lane) while 8 MFMAs consume the
// current ones.  Operand values toggle like the real planes, which lowers
// the sustained clock well below the near-constant operands of k_mfma_peak.
typedef __attribute__((address_space(3))) uint8_t lds_u8;
__device__ __forceinline__ v8i lds_frag(const uint8_t* base, int off) {
  const uint4 lo = *reinterpret_cast<const uint4*>(base + off);
  const uint4 hi = *reinterpret_cast<const uint4*>(base + off + 16);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}
__device__ __forceinline__ void digit_step(const uint8_t* L, int o, const v8i (&ca)[4],
                                           const v8i (&cb)[2], v8i (&na)[4], v8i (&nb)[2],
                                           v16f (&acc)[4][2]) {
  // o is a multiple of 32 below 65536; every offset stays inside the 64 KiB
#pragma unroll
  for (int x = 0; x < 4; ++x) na[x] = lds_frag(L, (o + 1024 * x) & 0xFFE0);
#pragma unroll
  for (int y = 0; y < 2; ++y) nb[y] = lds_frag(L, (o + 16384 + 1024 * y) & 0xFFE0);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ca[i], cb[j], acc[i][j], 0, 0, 0,
                                                                 0, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
}
__global__ void __launch_bounds__(512) k_mfma_digits(int iters, float* sink) {
  __shared__ __attribute__((aligned(16))) uint8_t L[65536];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  for (int i = t; i < 65536 / 4; i += 512) {
    uint32_t h = (uint32_t)i * 2654435761u ^ (uint32_t)blockIdx.x * 40503u, word = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      h = h * 1664525u + 1013904223u;
      const float d = (float)((int)((h >> 16) % 23u) - 11);
      word |= ((uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(d, 0.0f, 0, false) & 0xFFu) << (8 * b);
    }
    reinterpret_cast<uint32_t*>(L)[i] = word;
  }
  __syncthreads();
  v16f acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v16f{0.f};
  const int base = (w * 4096 + lane * 32) & 0xFFE0;
  v8i fa[4], fb[2], na[4], nb[2];
#pragma unroll
  for (int x = 0; x < 4; ++x) fa[x] = lds_frag(L, (base + 2048 * x) & 0xFFE0);
#pragma unroll
  for (int y = 0; y < 2; ++y) fb[y] = lds_frag(L, (base + 8192 + 2048 * y) & 0xFFE0);
  for (int it = 0; it < iters; it += 2) {
    digit_step(L, base + (it & 7) * 4096, fa, fb, na, nb, acc);
    digit_step(L, base + ((it + 1) & 7) * 4096, na, nb, fa, fb, acc);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) s += acc[i][j][e];
  if (s == 1.0e30f) sink[t] = s;   // keeps the MFMAs live; never true
}

int gfx950_ok() {
  int dev = 0;
  hipDeviceProp_t prop;
  if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess)
    return OZ2_E_DEVICE;
  return std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? OZ2_OK : OZ2_E_UNSUPPORTED;
}

int status(hipError_t e) { return e == hipSuccess ? OZ2_OK : OZ2_E_DEVICE; }

// One warm-up and one timed launch of an MFMA probe kernel (one 512-thread
// workgroup per CU, 8 waves x 8 MFMAs of 32x32x64 per iteration) on an
// internal stream; *tflops = FP8 TFLOP/s of the timed launch.
int time_mfma(void (*kern)(int, float*), int iters, double* tflops) {
  int st = gfx950_ok();
  if (st != OZ2_OK) return st;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return OZ2_E_DEVICE;
  float* sink = nullptr;
  hipStream_t s = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipMalloc(&sink, 512 * sizeof(float));
  if (e == hipSuccess) e = hipStreamCreate(&s);
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(kern, dim3(cus), dim3(512), 0, s, iters, sink);   // warm-up
    e = hipEventRecord(e0, s);
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(kern, dim3(cus), dim3(512), 0, s, iters, sink);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e == hipSuccess) {
    const double flop = 2.0 * 32 * 32 * 64 * 8.0 * iters * 8.0 * cus;   // 8 waves x 8 MFMAs x iters
    *tflops = flop / (ms * 1e-3) / 1e12;
  }
  if (e1) (void)hipEventDestroy(e1);
  if (e0) (void)hipEventDestroy(e0);
  if (s) (void)hipStreamDestroy(s);
  if (sink) (void)hipFree(sink);
  return status(e);
}

}  // namespace

extern "C" {

int ozaki2_probe_e4m3(const float* x, unsigned char* out, int n, void* stream) {
  if (n < 0 || (n > 0 && (!x || !out))) return OZ2_E_INVALID;
  if (n == 0) return OZ2_OK;
  int st = gfx950_ok();
  if (st != OZ2_OK) return st;
  hipLaunchKernelGGL(k_e4m3, dim3((n + 255) / 256), dim3(256), 0, (hipStream_t)stream, x, out, n);
  return status(hipGetLastError());
}

int ozaki2_probe_accum(const unsigned char* a, const unsigned char* b, int chain, float* out,
                       void* stream) {
  if (!a || !b || !out || chain < 1 || chain > (1 << 20)) return OZ2_E_INVALID;
  int st = gfx950_ok();
  if (st != OZ2_OK) return st;
  hipLaunchKernelGGL(k_accum, dim3(1), dim3(64), 0, (hipStream_t)stream, a, b, chain, out);
  return status(hipGetLastError());
}

int ozaki2_probe_copy(const void* src, void* dst, size_t bytes, void* stream) {
  if (bytes % 16 || ((uintptr_t)src % 16) || ((uintptr_t)dst % 16)) return OZ2_E_INVALID;
  if (bytes == 0) return OZ2_OK;
  if (!src || !dst) return OZ2_E_INVALID;
  int st = gfx950_ok();
  if (st != OZ2_OK) return st;
  const size_t n16 = bytes / 16;
  size_t blocks = (n16 + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(k_copy, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                     (const uint4*)src, (uint4*)dst, n16);
  return status(hipGetLastError());
}

int ozaki2_probe_mfma_peak(int iters, double* tflops) {
  if (iters < 1 || !tflops) return OZ2_E_INVALID;
  return time_mfma(k_mfma_peak, iters, tflops);
}

int ozaki2_probe_mfma_digits(int iters, double* tflops) {
  if (iters < 2 || iters % 2 || !tflops) return OZ2_E_INVALID;
  return time_mfma(k_mfma_digits, iters, tflops);
}

int ozaki2_probe_copy_peak(size_t bytes, int reps, double* gbs) {
  if (bytes < ((size_t)16 << 20) || bytes % 16 || reps < 1 || !gbs) return OZ2_E_INVALID;
  int st = gfx950_ok();
  if (st != OZ2_OK) return st;
  void *src = nullptr, *dst = nullptr;
  hipStream_t s = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipMalloc(&src, bytes);
  if (e == hipSuccess) e = hipMalloc(&dst, bytes);
  if (e == hipSuccess) e = hipMemset(src, 0x5A, bytes);
  if (e == hipSuccess) e = hipStreamCreate(&s);
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  auto copy = [&]() {
    return ozaki2_probe_copy(src, dst, bytes, s) == OZ2_OK ? hipSuccess : hipErrorLaunchFailure;
  };
  if (e == hipSuccess) e = copy();   // warm-up
  if (e == hipSuccess) e = hipEventRecord(e0, s);
  for (int i = 0; i < reps && e == hipSuccess; ++i) e = copy();
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e == hipSuccess) *gbs = 2.0 * (double)bytes * reps / (ms * 1e-3) / 1e9;
  if (e1) (void)hipEventDestroy(e1);
  if (e0) (void)hipEventDestroy(e0);
  if (s) (void)hipStreamDestroy(s);
  if (dst) (void)hipFree(dst);
  if (src) (void)hipFree(src);
  return status(e);
}

}  // extern "C"
