// The cross-term diagnostic of the error model (Appendix D: how much of the
// error's linear part the diagonal sum defining Phi leaves out).
//
// For a depth-1 plan whose workspace holds the encoding of A and B: with X_r,
// Y_r the fp32 combinations and dX_r = Xhat_r - X_r, dY_r = Yhat_r - Y_r their
// rounding residuals (Xhat_r the stored codes times their scales, exact in
// binary64), the part of sub-product r's error that is linear in the
// residuals is t_r = dX_r Y_r + X_r dY_r, and that of output block q is
// L_q = sum_r w[r, q] t_r.  Per batch element the kernels return
// |L|^2 = sum_q |L_q|^2 and diag = sum_{r, q} w[r, q]^2 |t_r|^2 in binary64;
// (|L|^2 - diag) / |L|^2 is the residual fraction.
//
//   1. resid_kernel<SIDE>: X_r (the encoder's combination: nonzero
//      coefficients in ascending block order, fp32 products and sums, no
//      fused multiply-add) and dX_r, both binary64, [batch][T][rows][k'];
//      the B side's rows are the columns of y_r (contracted axis last).
//      Codes and scales are read in whichever layout the plan keeps them.
//   2. cross_gemm_kernel: t_r = dX_r Y_r + X_r dY_r in binary64 (LDS tiles of
//      64 x 64 outputs, 4 x 4 per thread, contracted steps of 16).
//   3. cross_partials_kernel / cross_totals_kernel: L_q over the terms in
//      ascending order at every position, |L_q|^2 and the diagonal summed by a
//      fixed grid and a fixed tree (identical results run to run).
// Measurement infrastructure: not on the timed path.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace fmm {

namespace {

// exact value of an e4m3 code (codes 0x7F / 0xFF, NaN, are never stored)
__device__ __forceinline__ double e4m3_value(uint32_t code) {
  const uint32_t E = (code >> 3) & 15u, m = code & 7u;
  const double v = E == 0 ? (double)m * 0x1p-9 : (double)(8u + m) * ldexp(1.0, (int)E - 10);
  return (code & 0x80u) ? -v : v;
}

// code and scale of position (row, l) of term r, batch element bt, in the
// plan's layout (include/fmm8.h, FMM_LAYOUT_*)
__device__ __forceinline__ double decoded(const Problem &pb, const uint8_t *codes, const uint8_t *scales,
                                          int64_t rows, int64_t bt, int64_t r, int64_t row, int64_t l) {
  const int64_t plane = bt * pb.T + r;
  const int64_t kb = l / pb.block;
  uint32_t code;
  double s;
  if (pb.layout == FMM_LAYOUT_TILE256x64) {
    const int64_t t = row & 255, c = (l & 63) >> 4;
    code = codes[(((plane * (rows / 256) + row / 256) * (pb.kp / 64) + l / 64) * 256 + t) * 64 +
                 16 * (c ^ ((t >> 2) & 3)) + (l & 15)];
    const int64_t sbase = (plane * pb.kblocks + kb) * rows;
    if (pb.scale_bytes == 4) {
      s = (double)reinterpret_cast<const float *>(scales)[sbase + row];
    } else {
      const int64_t pos = (row & ~int64_t(255)) + 4 * (32 * (t >> 7) + (t & 31)) + ((t >> 5) & 3);
      s = ldexp(1.0, (int)scales[sbase + pos] - 127);
    }
  } else if (pb.layout == FMM_LAYOUT_TILE128x128) {
    const int64_t t = row & 127, c = (l & 127) >> 4;
    const int64_t tile = (plane * (rows / 128) + row / 128) * (pb.kp / 128) + l / 128;
    code = codes[(tile * 128 + t) * 128 + 16 * (c ^ (t & 7) ^ ((t >> 3) & 1)) + (l & 15)];
    if (pb.block == 16) {
      const int64_t b = (l & 127) >> 4;                      // record: blocks 0, 2, 4, 6, 1, 3, 5, 7
      s = ldexp(1.0, (int)scales[(tile * 128 + t) * 8 + 4 * (b & 1) + (b >> 1)] - 127);
    } else {
      const int64_t kk = (l & 127) >> 5;                     // block of 32 within the step
      const int64_t byte = pb.block == 32 ? (((kk & 1) << 1) | (kk >> 1)) : 0;   // record: blocks 0, 2, 1, 3
      s = ldexp(1.0, (int)scales[(tile * 128 + t) * 4 + byte] - 127);
    }
  } else {
    code = codes[(plane * rows + row) * pb.kp + l];
    const int64_t si = (plane * rows + row) * pb.kblocks + kb;
    s = pb.scale_bytes == 4 ? (double)reinterpret_cast<const float *>(scales)[si]
                            : ldexp(1.0, (int)scales[si] - 127);
  }
  return e4m3_value(code) * s;
}

// X and dX of one side, one thread per (row, l) of term blockIdx.y, batch blockIdx.z
template <int SIDE>
__global__ __launch_bounds__(256) void resid_kernel(const float *__restrict__ src, const int32_t *__restrict__ off,
                                                    const CoefEntry *__restrict__ ent, const uint8_t *__restrict__ codes,
                                                    const uint8_t *__restrict__ scales, double *__restrict__ X,
                                                    double *__restrict__ D, Problem pb) {
  const int64_t rows = SIDE == 0 ? pb.mp : pb.np;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * pb.kp) return;
  const int64_t r = blockIdx.y, bt = blockIdx.z;
  const int64_t row = idx / pb.kp, l = idx - row * pb.kp;
  // A: block (P, Q) = rows P m' + row, columns Q k' + l of A;
  // B: block (J, K) = rows J k' + l, columns K n' + row of B
  const float *base = SIDE == 0 ? src + bt * pb.M * pb.K : src + bt * pb.K * pb.N;
  float x = 0.0f;
  bool first = true;
  for (int e = off[r]; e < off[r + 1]; ++e) {
    const int b = ent[e].block;
    const int64_t P = b / pb.nsplit, Q = b % pb.nsplit;
    const float a = SIDE == 0 ? base[(P * pb.mp + row) * pb.K + Q * pb.kp + l]
                              : base[(P * pb.kp + l) * pb.N + Q * pb.np + row];
    const float prod = __fmul_rn(ent[e].coef, a);
    x = first ? prod : __fadd_rn(x, prod);
    first = false;
  }
  const double xh = decoded(pb, codes, scales, rows, bt, r, row, l);
  const int64_t o = ((bt * pb.T + r) * rows + row) * pb.kp + l;
  X[o] = (double)x;
  D[o] = xh - (double)x;
}

constexpr int GT = 64, GK = 16;

// t_r = dX_r Y_r + X_r dY_r: rows p of the A side, rows q of the B side (both
// with the contracted axis last); grid (tiles, T, batch)
__global__ __launch_bounds__(256) void cross_gemm_kernel(const double *__restrict__ XA, const double *__restrict__ DA,
                                                         const double *__restrict__ XB, const double *__restrict__ DB,
                                                         double *__restrict__ Tr, Problem pb, int64_t tiles_n) {
  __shared__ double xa[GK][GT + 1], da[GK][GT + 1], xb[GK][GT + 1], db[GK][GT + 1];
  const int t = threadIdx.x;
  const int64_t r = blockIdx.y, bt = blockIdx.z;
  const int64_t p0 = (blockIdx.x / tiles_n) * GT, q0 = (blockIdx.x % tiles_n) * GT;
  const int64_t pa = (bt * pb.T + r) * pb.mp, pbb = (bt * pb.T + r) * pb.np;
  const int tx = t % 16, ty = t / 16;
  double acc[4][4] = {};
  for (int64_t k0 = 0; k0 < pb.kp; k0 += GK) {
    for (int e = t; e < GT * GK; e += 256) {
      const int rr = e / GK, kk = e % GK;
      const int64_t k = k0 + kk;
      const int64_t p = p0 + rr, q = q0 + rr;
      const bool ka = k < pb.kp;
      xa[kk][rr] = (ka && p < pb.mp) ? XA[(pa + p) * pb.kp + k] : 0.0;
      da[kk][rr] = (ka && p < pb.mp) ? DA[(pa + p) * pb.kp + k] : 0.0;
      xb[kk][rr] = (ka && q < pb.np) ? XB[(pbb + q) * pb.kp + k] : 0.0;
      db[kk][rr] = (ka && q < pb.np) ? DB[(pbb + q) * pb.kp + k] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GK; ++kk) {
      double a0[4], a1[4], b0[4], b1[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a0[i] = da[kk][ty + 16 * i];
        a1[i] = xa[kk][ty + 16 * i];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        b0[j] = xb[kk][tx + 16 * j];
        b1[j] = db[kk][tx + 16 * j];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fma(a1[i], b1[j], fma(a0[i], b0[j], acc[i][j]));
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t p = p0 + ty + 16 * i, q = q0 + tx + 16 * j;
      if (p < pb.mp && q < pb.np) Tr[((bt * pb.T + r) * pb.mp + p) * pb.np + q] = acc[i][j];
    }
}

constexpr int kThreadsC = 256;
constexpr int kPartialsC = 512;   // partials per batch element

__device__ __forceinline__ void tree_sum2(double *s0, double *s1, int t) {
  for (int w = kThreadsC / 2; w > 0; w >>= 1) {
    if (t < w) {
      s0[t] += s0[t + w];
      s1[t] += s1[t + w];
    }
    __syncthreads();
  }
}

// grid (kPartialsC, batch): at every position of the m' x n' grid,
// L_q = sum_r w[r][q] t_r (ascending r), |L_q|^2 and sum_r (sum_q w[r][q]^2) t_r^2
__global__ __launch_bounds__(kThreadsC) void cross_partials_kernel(const double *__restrict__ Tr,
                                                                   const float *__restrict__ w,
                                                                   double *__restrict__ part, Problem pb) {
  __shared__ double s0[kThreadsC], s1[kThreadsC];
  const int t = threadIdx.x;
  const int64_t bt = blockIdx.y;
  const int64_t plane = pb.mp * pb.np;
  const int T = (int)pb.T;
  double wr[kMaxRank][4], w2[kMaxRank];
#pragma unroll
  for (int r = 0; r < kMaxRank; ++r) {
    w2[r] = 0.0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      wr[r][q] = (double)w[4 * r + q];    // zero-padded table
      w2[r] += wr[r][q] * wr[r][q];
    }
  }
  double l2 = 0.0, dg = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * kThreadsC + t; i < plane; i += (int64_t)kPartialsC * kThreadsC) {
    double L[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int r = 0; r < kMaxRank; ++r) {
      if (r < T) {
        const double v = Tr[(bt * pb.T + r) * plane + i];
#pragma unroll
        for (int q = 0; q < 4; ++q) L[q] = fma(wr[r][q], v, L[q]);
        dg = fma(w2[r], v * v, dg);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) l2 = fma(L[q], L[q], l2);
  }
  s0[t] = l2;
  s1[t] = dg;
  __syncthreads();
  tree_sum2(s0, s1, t);
  if (t == 0) {
    part[(bt * kPartialsC + blockIdx.x) * 2] = s0[0];
    part[(bt * kPartialsC + blockIdx.x) * 2 + 1] = s1[0];
  }
}

__global__ __launch_bounds__(kThreadsC) void cross_totals_kernel(const double *__restrict__ part,
                                                                 double *__restrict__ out) {
  __shared__ double s0[kThreadsC], s1[kThreadsC];
  const int t = threadIdx.x;
  const int64_t bt = blockIdx.x;
  double a = 0.0, b = 0.0;
  for (int i = t; i < kPartialsC; i += kThreadsC) {
    a += part[(bt * kPartialsC + i) * 2];
    b += part[(bt * kPartialsC + i) * 2 + 1];
  }
  s0[t] = a;
  s1[t] = b;
  __syncthreads();
  tree_sum2(s0, s1, t);
  if (t == 0) {
    out[2 * bt] = s0[0];
    out[2 * bt + 1] = s1[0];
  }
}

// scratch sections, 256-byte aligned: XA, DA, XB, DB, t, partials
struct CrossScratch {
  size_t xa, da, xb, db, tr, part, total;
};

CrossScratch cross_layout(const Problem &pb) {
  auto al = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t B = (size_t)pb.batch, T = (size_t)pb.T;
  CrossScratch c;
  size_t off = 0;
  c.xa = off; off = al(off + B * T * pb.mp * pb.kp * 8);
  c.da = off; off = al(off + B * T * pb.mp * pb.kp * 8);
  c.xb = off; off = al(off + B * T * pb.np * pb.kp * 8);
  c.db = off; off = al(off + B * T * pb.np * pb.kp * 8);
  c.tr = off; off = al(off + B * T * pb.mp * pb.np * 8);
  c.part = off; off = al(off + B * kPartialsC * 2 * 8);
  c.total = off;
  return c;
}

}  // namespace

size_t cross_terms_scratch_bytes(const Problem &pb) { return cross_layout(pb).total; }

int launch_cross_terms(const Problem &pb, const DeviceTables &tab, const float *A, const float *B,
                       const uint8_t *ws, const Workspace &wl, double *out, void *scratch, void *stream) {
  if (pb.batch == 0) return hipSuccess;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const CrossScratch cl = cross_layout(pb);
  uint8_t *s = reinterpret_cast<uint8_t *>(scratch);
  double *XA = reinterpret_cast<double *>(s + cl.xa), *DA = reinterpret_cast<double *>(s + cl.da);
  double *XB = reinterpret_cast<double *>(s + cl.xb), *DB = reinterpret_cast<double *>(s + cl.db);
  double *Tr = reinterpret_cast<double *>(s + cl.tr), *part = reinterpret_cast<double *>(s + cl.part);
  const int64_t plane = pb.mp * pb.np;
  if (plane > 0 && pb.kp > 0) {
    const dim3 ga((unsigned)((pb.mp * pb.kp + 255) / 256), (unsigned)pb.T, (unsigned)pb.batch);
    hipLaunchKernelGGL(resid_kernel<0>, ga, dim3(256), 0, st, A, tab.a_off, tab.a_ent, ws + wl.a_codes,
                       ws + wl.a_scales, XA, DA, pb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 gb((unsigned)((pb.np * pb.kp + 255) / 256), (unsigned)pb.T, (unsigned)pb.batch);
    hipLaunchKernelGGL(resid_kernel<1>, gb, dim3(256), 0, st, B, tab.b_off, tab.b_ent, ws + wl.b_codes,
                       ws + wl.b_scales, XB, DB, pb);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (plane > 0) {   // (k' = 0: no contracted step, every t_r written as zero)
    const int64_t tn = (pb.np + GT - 1) / GT, tm = (pb.mp + GT - 1) / GT;
    hipLaunchKernelGGL(cross_gemm_kernel, dim3((unsigned)(tm * tn), (unsigned)pb.T, (unsigned)pb.batch),
                       dim3(256), 0, st, XA, DA, XB, DB, Tr, pb, tn);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(cross_partials_kernel, dim3(kPartialsC, (unsigned)pb.batch), dim3(kThreadsC), 0, st, Tr,
                     tab.w_inner, part, pb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(cross_totals_kernel, dim3((unsigned)pb.batch), dim3(kThreadsC), 0, st, part, out);
  return hipGetLastError();
}

}  // namespace fmm
