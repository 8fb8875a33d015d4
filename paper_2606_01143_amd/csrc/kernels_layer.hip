// Token-wise operations of a decoder layer: RMSNorm, rotary embedding and
// SwiGLU, forward and backward.  Each streams its tensors once with 16-byte
// accesses (HBM bound); reductions of a row stay inside one workgroup.
#include <math.h>

#include "launch.hpp"

namespace spr {

namespace {
constexpr int kRowThreads = 256;

__device__ __forceinline__ void load8(const bf16* p, float (&v)[8]) {
  const bf16x8 x = *(const bf16x8*)p;
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = (float)x[j];
}
__device__ __forceinline__ void store8(bf16* p, const float (&v)[8]) {
  bf16x8 x;
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = (bf16)v[j];
  *(bf16x8*)p = x;
}

// sum over the workgroup, the same value returned to every thread
__device__ float block_sum(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < kRowThreads / 64; ++i) s += red[i];
  return s;
}
}  // namespace

// one workgroup per row; each thread holds up to 8 chunks of 8 values
constexpr int kMaxChunks = 8;

__global__ __launch_bounds__(kRowThreads) void rmsnorm_fwd_kernel(const bf16* __restrict__ x, bf16* __restrict__ y,
                                                                  float* __restrict__ rstd, int width, float eps) {
  __shared__ float red[kRowThreads / 64];
  const long row = blockIdx.x;
  const bf16* xr = x + row * width;
  const int chunks = width / 8;
  float v[kMaxChunks][8];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < kMaxChunks; ++c) {
    const int ch = threadIdx.x + c * kRowThreads;
    if (ch < chunks) {
      load8(xr + 8 * ch, v[c]);
#pragma unroll
      for (int j = 0; j < 8; ++j) ss = fmaf(v[c][j], v[c][j], ss);
    }
  }
  const float r = rsqrtf(block_sum(ss, red) / (float)width + eps);
#pragma unroll
  for (int c = 0; c < kMaxChunks; ++c) {
    const int ch = threadIdx.x + c * kRowThreads;
    if (ch < chunks) {
      float o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = v[c][j] * r;
      store8(y + row * width + 8 * ch, o);
    }
  }
  if (threadIdx.x == 0) rstd[row] = r;
}

__global__ __launch_bounds__(kRowThreads) void rmsnorm_bwd_kernel(const bf16* __restrict__ x,
                                                                  const float* __restrict__ rstd,
                                                                  const bf16* __restrict__ dy,
                                                                  const bf16* __restrict__ add, bf16* __restrict__ dx,
                                                                  int width) {
  __shared__ float red[kRowThreads / 64];
  const long row = blockIdx.x;
  const int chunks = width / 8;
  const float r = rstd[row];
  float xv[kMaxChunks][8], gv[kMaxChunks][8];
  float dot = 0.f;
#pragma unroll
  for (int c = 0; c < kMaxChunks; ++c) {
    const int ch = threadIdx.x + c * kRowThreads;
    if (ch < chunks) {
      load8(x + row * width + 8 * ch, xv[c]);
      load8(dy + row * width + 8 * ch, gv[c]);
#pragma unroll
      for (int j = 0; j < 8; ++j) dot = fmaf(gv[c][j], xv[c][j], dot);
    }
  }
  // dx = r dy - r^3 x mean(dy x)
  const float k3 = r * r * r * block_sum(dot, red) / (float)width;
#pragma unroll
  for (int c = 0; c < kMaxChunks; ++c) {
    const int ch = threadIdx.x + c * kRowThreads;
    if (ch < chunks) {
      float o[8], a[8];
      if (add)
        load8(add + row * width + 8 * ch, a);
      else
#pragma unroll
        for (int j = 0; j < 8; ++j) a[j] = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = r * gv[c][j] - k3 * xv[c][j] + a[j];
      store8(dx + row * width + 8 * ch, o);
    }
  }
}

// one workgroup per token; thread (head, j) rotates the pair (j, j + d/2)
__global__ __launch_bounds__(kRowThreads) void rope_kernel(const bf16* __restrict__ x, bf16* __restrict__ y,
                                                           int heads, int d, int pos0, double theta, float sign) {
  const long t = blockIdx.x;
  const int half = d / 2;
  const double pos = (double)(pos0 + t);
  for (int i = threadIdx.x; i < heads * half; i += kRowThreads) {
    const int h = i / half, j = i % half;
    // angle in fp64, reduced to [-pi, pi] before the fp32 sine and cosine
    double ang = pos * pow(theta, -2.0 * (double)j / (double)d);
    ang = remainder(ang, 2.0 * M_PI);
    float sn, cs;
    sincosf((float)ang, &sn, &cs);
    sn *= sign;
    const long base = (t * heads + h) * d;
    const float a = (float)x[base + j], b = (float)x[base + j + half];
    y[base + j] = (bf16)(a * cs - b * sn);
    y[base + j + half] = (bf16)(b * cs + a * sn);
  }
}

__global__ __launch_bounds__(256) void swiglu_fwd_kernel(const bf16* __restrict__ g, const bf16* __restrict__ u,
                                                         bf16* __restrict__ m, long n8) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  float gv[8], uv[8], o[8];
  load8(g + 8 * i, gv);
  load8(u + 8 * i, uv);
#pragma unroll
  for (int j = 0; j < 8; ++j) o[j] = gv[j] / (1.f + __expf(-gv[j])) * uv[j];
  store8(m + 8 * i, o);
}

__global__ __launch_bounds__(256) void swiglu_bwd_kernel(const bf16* __restrict__ g, const bf16* __restrict__ u,
                                                         const bf16* __restrict__ dm, bf16* __restrict__ dg,
                                                         bf16* __restrict__ du, long n8) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  float gv[8], uv[8], dv[8], og[8], ou[8];
  load8(g + 8 * i, gv);
  load8(u + 8 * i, uv);
  load8(dm + 8 * i, dv);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float s = 1.f / (1.f + __expf(-gv[j]));
    const float silu = gv[j] * s;
    og[j] = dv[j] * uv[j] * s * (1.f + gv[j] * (1.f - s));
    ou[j] = dv[j] * silu;
  }
  store8(dg + 8 * i, og);
  store8(du + 8 * i, ou);
}

hipError_t launch_rmsnorm_fwd(int rows, int width, float eps, const void* x, void* y, float* rstd, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  ProfileScope ps("rmsnorm_fwd", st);
  hipLaunchKernelGGL(rmsnorm_fwd_kernel, dim3(rows), dim3(kRowThreads), 0, st, (const bf16*)x, (bf16*)y, rstd, width,
                     eps);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_bwd(int rows, int width, const void* x, const float* rstd, const void* dy, const void* add,
                              void* dx, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  ProfileScope ps("rmsnorm_bwd", st);
  hipLaunchKernelGGL(rmsnorm_bwd_kernel, dim3(rows), dim3(kRowThreads), 0, st, (const bf16*)x, rstd,
                     (const bf16*)dy, (const bf16*)add, (bf16*)dx, width);
  return hipGetLastError();
}

hipError_t launch_rope(int tokens, int heads, int d, int pos0, double theta, const void* x, void* y, bool inverse,
                       hipStream_t st) {
  if (tokens == 0) return hipSuccess;
  ProfileScope ps(inverse ? "rope_bwd" : "rope_fwd", st);
  hipLaunchKernelGGL(rope_kernel, dim3(tokens), dim3(kRowThreads), 0, st, (const bf16*)x, (bf16*)y, heads, d, pos0,
                     theta, inverse ? -1.f : 1.f);
  return hipGetLastError();
}

hipError_t launch_swiglu_fwd(long n, const void* g, const void* u, void* m, hipStream_t st) {
  const long n8 = n / 8;
  if (n8 == 0) return hipSuccess;
  ProfileScope ps("swiglu_fwd", st);
  hipLaunchKernelGGL(swiglu_fwd_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, st, (const bf16*)g,
                     (const bf16*)u, (bf16*)m, n8);
  return hipGetLastError();
}

hipError_t launch_swiglu_bwd(long n, const void* g, const void* u, const void* dm, void* dg, void* du,
                             hipStream_t st) {
  const long n8 = n / 8;
  if (n8 == 0) return hipSuccess;
  ProfileScope ps("swiglu_bwd", st);
  hipLaunchKernelGGL(swiglu_bwd_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, st, (const bf16*)g,
                     (const bf16*)u, (const bf16*)dm, (bf16*)dg, (bf16*)du, n8);
  return hipGetLastError();
}

}  // namespace spr
