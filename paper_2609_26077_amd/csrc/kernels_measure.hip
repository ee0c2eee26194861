// Error measurement (Appendix E.2: relative error against an fp64 product)
// and the standalone e4m3 codec.
//
// reference_f64_kernel: C_ref = A B in binary64 from fp32 operands; LDS-tiled,
//   64 x 64 outputs per workgroup, 4 x 4 per thread, K steps of 16.
//   Measurement infrastructure: not on the timed path.
// error partials / totals: per product, sum (C - C_ref)^2 and sum C_ref^2 in
//   binary64 by a fixed grid of workgroups (each a fixed-order strided sum and
//   a fixed LDS tree), then one workgroup per product adds the partials in
//   index order.  No atomics, so results are identical run to run.
// The allocation-free form of the reduction keeps its partials in `scratch`,
//   a static device array of this file (one copy per device).
#include <hip/hip_runtime.h>

#include <mutex>

#include "device.h"
#include "internal.h"

namespace fmm {

namespace {

constexpr int RT = 64, RK = 16;

__global__ __launch_bounds__(256) void reference_f64_kernel(const float *__restrict__ A,
                                                            const float *__restrict__ B,
                                                            double *__restrict__ C, int64_t M,
                                                            int64_t K, int64_t N, int64_t tiles_n) {
  __shared__ double la[RK][RT + 1];
  __shared__ double lb[RK][RT + 1];
  const int t = threadIdx.x;
  const int64_t bt = blockIdx.z;
  const int64_t m0 = (blockIdx.x / tiles_n) * RT, n0 = (blockIdx.x % tiles_n) * RT;
  const float *Ab = A + bt * M * K;
  const float *Bb = B + bt * K * N;
  const int tx = t % 16, ty = t / 16;   // 4 x 4 outputs at rows ty + 16 i, cols tx + 16 j
  double acc[4][4] = {};
  for (int64_t k0 = 0; k0 < K; k0 += RK) {
    // A tile: 64 rows x 16 k; B tile: 16 k x 64 cols (1024 elements each)
    for (int e = t; e < RT * RK; e += 256) {
      const int r = e / RK, kk = e % RK;
      const int64_t gm = m0 + r, gk = k0 + kk;
      la[kk][r] = (gm < M && gk < K) ? (double)Ab[gm * K + gk] : 0.0;
      const int kb = e / RT, c = e % RT;
      const int64_t gk2 = k0 + kb, gn = n0 + c;
      lb[kb][c] = (gk2 < K && gn < N) ? (double)Bb[gk2 * N + gn] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < RK; ++kk) {
      double a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = la[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = lb[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fma(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t gm = m0 + ty + 16 * i, gn = n0 + tx + 16 * j;
      if (gm < M && gn < N) C[bt * M * N + gm * N + gn] = acc[i][j];
    }
}

constexpr int kRedThreads = 256;
constexpr int kRedBlocks = 512;   // partials per product

// Partials of the allocation-free reduction: kStaticErrorBatch products of
// kRedBlocks (err2, ref2) pairs, 8 MiB.  Every partial is written before it
// is read, so nothing needs clearing between calls.
static __device__ __align__(256) double scratch[kStaticErrorBatch * kRedBlocks * 2];

__device__ __forceinline__ void tree_sum2(double *s0, double *s1, int t) {
  for (int w = kRedThreads / 2; w > 0; w >>= 1) {
    if (t < w) {
      s0[t] += s0[t + w];
      s1[t] += s1[t + w];
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(kRedThreads) void error_partials_kernel(const float *__restrict__ C,
                                                                     const double *__restrict__ Cref,
                                                                     double *__restrict__ part,
                                                                     int64_t MN) {
  __shared__ double s0[kRedThreads], s1[kRedThreads];
  const int t = threadIdx.x;
  const int64_t bt = blockIdx.y;
  const float *c = C + bt * MN;
  const double *r = Cref + bt * MN;
  double e2 = 0.0, r2 = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * kRedThreads + t; i < MN; i += (int64_t)kRedBlocks * kRedThreads) {
    const double ref = r[i];
    const double d = (double)c[i] - ref;
    e2 = fma(d, d, e2);
    r2 = fma(ref, ref, r2);
  }
  s0[t] = e2;
  s1[t] = r2;
  __syncthreads();
  tree_sum2(s0, s1, t);
  if (t == 0) {
    part[(bt * kRedBlocks + blockIdx.x) * 2] = s0[0];
    part[(bt * kRedBlocks + blockIdx.x) * 2 + 1] = s1[0];
  }
}

__global__ __launch_bounds__(kRedThreads) void error_totals_kernel(const double *__restrict__ part,
                                                                   double *__restrict__ out) {
  __shared__ double s0[kRedThreads], s1[kRedThreads];
  const int t = threadIdx.x;
  const int64_t bt = blockIdx.x;
  double e2 = 0.0, r2 = 0.0;
  for (int i = t; i < kRedBlocks; i += kRedThreads) {
    e2 += part[(bt * kRedBlocks + i) * 2];
    r2 += part[(bt * kRedBlocks + i) * 2 + 1];
  }
  s0[t] = e2;
  s1[t] = r2;
  __syncthreads();
  tree_sum2(s0, s1, t);
  if (t == 0) {
    out[2 * bt] = s0[0];
    out[2 * bt + 1] = s1[0];
  }
}

__global__ __launch_bounds__(256) void e4m3_quantize_kernel(const float *__restrict__ in,
                                                            uint8_t *__restrict__ out, int64_t n) {
  const int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i4 + 3 < n) {
    const float4 v = *reinterpret_cast<const float4 *>(in + i4);
    *reinterpret_cast<uint32_t *>(out + i4) = dev::e4m3_pack4(v.x, v.y, v.z, v.w);
  } else if (i4 < n) {
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    for (int k = 0; i4 + k < n; ++k) v[k] = in[i4 + k];
    const uint32_t w = dev::e4m3_pack4(v[0], v[1], v[2], v[3]);
    for (int k = 0; i4 + k < n; ++k) out[i4 + k] = (uint8_t)(w >> (8 * k));
  }
}

// The cast of the power-of-two scale rules: codes of in[i] / s, s = 2^e,
// through the routine the encoder applies to every block with an E8M0 scale.
__global__ __launch_bounds__(256) void e4m3_quantize_pow2_kernel(const float *__restrict__ in,
                                                                 uint8_t *__restrict__ out, int64_t n,
                                                                 float s) {
  const int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i4 + 3 < n) {
    const float4 v = *reinterpret_cast<const float4 *>(in + i4);
    *reinterpret_cast<uint32_t *>(out + i4) = dev::e4m3_pack4_pow2(v.x, v.y, v.z, v.w, s);
  } else if (i4 < n) {
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    for (int k = 0; i4 + k < n; ++k) v[k] = in[i4 + k];
    const uint32_t w = dev::e4m3_pack4_pow2(v[0], v[1], v[2], v[3], s);
    for (int k = 0; i4 + k < n; ++k) out[i4 + k] = (uint8_t)(w >> (8 * k));
  }
}

}  // namespace

int launch_reference_f64(int64_t batch, int64_t M, int64_t K, int64_t N, const float *A,
                         const float *B, double *Cref, void *stream) {
  if (batch == 0 || M == 0 || N == 0) return hipSuccess;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int64_t tm = (M + RT - 1) / RT, tn = (N + RT - 1) / RT;
  hipLaunchKernelGGL(reference_f64_kernel, dim3((unsigned)(tm * tn), 1, (unsigned)batch), dim3(256),
                     0, st, A, B, Cref, M, K, N, tn);
  return hipGetLastError();
}

size_t error_stats_scratch_bytes(int64_t batch, int64_t, int64_t) {
  return (size_t)batch * kRedBlocks * 2 * sizeof(double);
}

int launch_error_stats(int64_t batch, int64_t M, int64_t N, const float *C, const double *Cref,
                       double *out, void *scratch, void *stream) {
  if (batch == 0) return hipSuccess;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  double *part = reinterpret_cast<double *>(scratch);
  hipLaunchKernelGGL(error_partials_kernel, dim3(kRedBlocks, (unsigned)batch), dim3(kRedThreads), 0,
                     st, C, Cref, part, M * N);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(error_totals_kernel, dim3((unsigned)batch), dim3(kRedThreads), 0, st, part, out);
  return hipGetLastError();
}

// The device address of `scratch` on the current device, looked up once per
// device (each device holds its own copy of the array at its own address).
// In host code the array's name is only a stand-in for the symbol, never an
// address a kernel may be given.
int static_error_scratch(void **ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

int launch_e4m3_quantize(const float *in, uint8_t *out, int64_t n, void *stream) {
  if (n == 0) return hipSuccess;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int64_t groups = (n + 3) / 4;
  hipLaunchKernelGGL(e4m3_quantize_kernel, dim3((unsigned)((groups + 255) / 256)), dim3(256), 0, st,
                     in, out, n);
  return hipGetLastError();
}

int launch_e4m3_quantize_pow2(const float *in, uint8_t *out, int64_t n, int e, void *stream) {
  if (n == 0) return hipSuccess;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int64_t groups = (n + 3) / 4;
  const uint32_t sbits = (uint32_t)(e + 127) << 23;   // 2^e, e in [-126, 127]
  float s;
  __builtin_memcpy(&s, &sbits, 4);
  hipLaunchKernelGGL(e4m3_quantize_pow2_kernel, dim3((unsigned)((groups + 255) / 256)), dim3(256), 0, st,
                     in, out, n, s);
  return hipGetLastError();
}

}  // namespace fmm
