// MoE router auxiliary-loss accounting under prefix reuse (paper Sec. 3.5,
// Sec. 4.6, App. B): multiplicity-weighted expert counts C_e, probability
// mass R_e and token total M, the Switch-style loss, and the router
// probability gradient.
//
// Everything here streams the [tokens, E] probability matrix once (HBM
// bound).  Reductions run in a fixed order so that results are bitwise
// reproducible: per-block partials in fp64 / int64, then one pass that adds
// the partials of all blocks in block order into the statistics.
#include <stdint.h>

#include <algorithm>

#include "launch.hpp"

namespace spr {

namespace {
constexpr int kMoeThreads = 256;

__device__ __forceinline__ long long token_mult(int u, int mult, const int* mu) {
  return mu != nullptr ? (long long)mu[u] : (long long)mult;
}
}  // namespace

// Block b takes tokens [b chunk, (b + 1) chunk).  Counts go through an LDS
// histogram (64-bit integer adds, exact); the probability mass is summed per
// thread over a strided subset of rows in fp64 (4 experts per thread, one
// 16-byte load per row), then the rows' partials are added in row order.
__global__ __launch_bounds__(kMoeThreads) void moe_partial_kernel(
    const float* __restrict__ p, const int* __restrict__ r, int n, int E, int k, int mult,
    const int* __restrict__ mu, int chunk, double* __restrict__ part_mass,
    long long* __restrict__ part_count, long long* __restrict__ part_tot) {
  __shared__ unsigned long long hist[1024];
  __shared__ double red[kMoeThreads * 4];
  __shared__ unsigned long long inval, tot;
  const int tid = threadIdx.x, b = blockIdx.x;
  const int u0 = b * chunk, u1 = min(n, u0 + chunk);
  for (int e = tid; e < E; e += kMoeThreads) hist[e] = 0;
  if (tid == 0) {
    inval = 0;
    tot = 0;
  }
  __syncthreads();
  // selected experts: pairs (u, j) of the chunk, contiguous in r
  const int npairs = (u1 - u0) * k;
  for (int i = tid; i < npairs; i += kMoeThreads) {
    const int u = u0 + i / k;
    const int e = r[(size_t)u0 * k + i];
    const long long m = token_mult(u, mult, mu);
    if (e >= 0 && e < E)
      atomicAdd(&hist[e], (unsigned long long)m);
    else
      atomicAdd(&inval, 1ull);
  }
  // multiplicity total of the chunk
  for (int u = u0 + tid; u < u1; u += kMoeThreads) atomicAdd(&tot, (unsigned long long)token_mult(u, mult, mu));
  // probability mass: cols threads per row, rows_par rows at a time
  const int cols = E / 4, rows_par = kMoeThreads / cols;
  const int tc = tid % cols, tr = tid / cols;
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
  if (tr < rows_par) {
    // eight rows' loads in flight before their products are added (in row order)
    constexpr int kRows = 8;
    for (int ub = u0 + tr; ub < u1; ub += kRows * rows_par) {
      float4 v[kRows];
      double m[kRows];
#pragma unroll
      for (int q = 0; q < kRows; ++q) {
        const int u = ub + q * rows_par;
        const bool in = u < u1;
        v[q] = in ? *(const float4*)(p + (size_t)u * E + 4 * tc) : make_float4(0.f, 0.f, 0.f, 0.f);
        m[q] = in ? (double)token_mult(u, mult, mu) : 0.0;
      }
#pragma unroll
      for (int q = 0; q < kRows; ++q) {
        a0 = fma(m[q], (double)v[q].x, a0);
        a1 = fma(m[q], (double)v[q].y, a1);
        a2 = fma(m[q], (double)v[q].z, a2);
        a3 = fma(m[q], (double)v[q].w, a3);
      }
    }
  }
  red[4 * tid + 0] = a0;
  red[4 * tid + 1] = a1;
  red[4 * tid + 2] = a2;
  red[4 * tid + 3] = a3;
  __syncthreads();
  double* pm = part_mass + (size_t)b * E;
  long long* pc = part_count + (size_t)b * E;
  for (int e = tid; e < E; e += kMoeThreads) {
    const int c = e / 4, q = e % 4;
    double s = 0.0;
    for (int row = 0; row < rows_par; ++row) s += red[4 * (row * cols + c) + q];
    pm[e] = s;
    pc[e] = (long long)hist[e];
  }
  if (tid == 0) {
    part_tot[2 * b] = (long long)tot;
    part_tot[2 * b + 1] = (long long)inval;
  }
}

// stats += the partials of blocks 0 .. nb - 1.  Block e < E owns expert e,
// block E the totals; thread t adds the partials of blocks t, t + 256, ...
// in order, then a fixed-shape tree adds the threads' sums.
__global__ __launch_bounds__(kMoeThreads) void moe_reduce_kernel(const double* __restrict__ part_mass,
                                                                 const long long* __restrict__ part_count,
                                                                 const long long* __restrict__ part_tot,
                                                                 int nb, int E, unsigned char* stats) {
  __shared__ double rm[kMoeThreads];
  __shared__ long long rc[kMoeThreads];
  const int tid = threadIdx.x, e = blockIdx.x;
  double s = 0.0;
  long long c = 0;
  if (e < E) {
    for (int b = tid; b < nb; b += kMoeThreads) {
      s += part_mass[(size_t)b * E + e];
      c += part_count[(size_t)b * E + e];
    }
  } else {
    long long inv = 0;
    for (int b = tid; b < nb; b += kMoeThreads) {
      c += part_tot[2 * b];
      inv += part_tot[2 * b + 1];
    }
    s = (double)inv;  // exact: far below 2^53
  }
  rm[tid] = s;
  rc[tid] = c;
  __syncthreads();
  for (int h = kMoeThreads / 2; h > 0; h >>= 1) {
    if (tid < h) {
      rm[tid] += rm[tid + h];
      rc[tid] += rc[tid + h];
    }
    __syncthreads();
  }
  if (tid != 0) return;
  long long* count = (long long*)stats;
  double* mass = (double*)(stats + 8 * (size_t)E);
  long long* total = (long long*)(stats + 16 * (size_t)E);
  if (e < E) {
    count[e] += rc[0];
    mass[e] += rm[0];
  } else {
    total[0] += rc[0];
    total[1] += (long long)rm[0];
  }
}

// f_e = C_e / (k M), P_e = R_e / M, L = coef E sum_e f_e P_e (one block,
// tree reduction in a fixed order).
__global__ __launch_bounds__(kMoeThreads) void moe_loss_kernel(const unsigned char* stats, int E, int k,
                                                               double coef, double* f, double* pe,
                                                               double* loss) {
  __shared__ double red[kMoeThreads];
  const long long* count = (const long long*)stats;
  const double* mass = (const double*)(stats + 8 * (size_t)E);
  const long long total = *(const long long*)(stats + 16 * (size_t)E);
  const int tid = threadIdx.x;
  double acc = 0.0;
  for (int e = tid; e < E; e += kMoeThreads) {
    const double fe = total > 0 ? (double)count[e] / ((double)k * (double)total) : 0.0;
    const double pv = total > 0 ? mass[e] / (double)total : 0.0;
    if (f) f[e] = fe;
    if (pe) pe[e] = pv;
    acc = fma(fe, pv, acc);
  }
  red[tid] = acc;
  __syncthreads();
  for (int s = kMoeThreads / 2; s > 0; s >>= 1) {
    if (tid < s) red[tid] += red[tid + s];
    __syncthreads();
  }
  if (tid == 0) loss[0] = coef * (double)E * red[0];
}

// dp[u, e] = upstream coef E f_e m_u / M, 4 experts per thread.
__global__ __launch_bounds__(kMoeThreads) void moe_grad_kernel(const unsigned char* stats, int E, int k,
                                                               double scale, int n, int mult,
                                                               const int* __restrict__ mu,
                                                               float* __restrict__ dp) {
  const long long* count = (const long long*)stats;
  const long long total = *(const long long*)(stats + 16 * (size_t)E);
  const int cols = E / 4;
  const long idx = (long)blockIdx.x * kMoeThreads + threadIdx.x;
  if (idx >= (long)n * cols) return;
  const int u = (int)(idx / cols), c = (int)(idx % cols);
  float4 out = make_float4(0.f, 0.f, 0.f, 0.f);
  if (total > 0) {
    // scale E f_e / M = scale E C_e / (k M^2)
    const double t = (double)total;
    const double w = scale * (double)E * (double)token_mult(u, mult, mu) / ((double)k * t * t);
    out.x = (float)(w * (double)count[4 * c + 0]);
    out.y = (float)(w * (double)count[4 * c + 1]);
    out.z = (float)(w * (double)count[4 * c + 2]);
    out.w = (float)(w * (double)count[4 * c + 3]);
  }
  *(float4*)(dp + (size_t)u * E + 4 * c) = out;
}

int moe_blocks(int n_tokens) {
  // 32 tokens per block (one load round trip per thread at E = 128), at
  // most 2048 partials per expert
  if (n_tokens <= 0) return 0;
  return std::min((n_tokens + 31) / 32, 2048);
}

size_t moe_workspace_bytes(int E, int n_tokens) {
  const size_t nb = (size_t)moe_blocks(n_tokens);
  return nb * (size_t)E * 16 + nb * 16;
}

hipError_t launch_moe_accumulate(const float* p, const int* r, int n, int E, int k, int mult,
                                 const int* mu, void* stats, void* ws, hipStream_t st) {
  const int nb = moe_blocks(n);
  if (nb == 0) return hipSuccess;
  const int chunk = (n + nb - 1) / nb;
  double* part_mass = (double*)ws;
  long long* part_count = (long long*)((unsigned char*)ws + (size_t)nb * E * 8);
  long long* part_tot = (long long*)((unsigned char*)ws + (size_t)nb * E * 16);
  {
    ProfileScope ps("moe_partial", st);
    hipLaunchKernelGGL(moe_partial_kernel, dim3(nb), dim3(kMoeThreads), 0, st, p, r, n, E, k, mult, mu, chunk,
                       part_mass, part_count, part_tot);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  ProfileScope pr("moe_reduce", st);
  hipLaunchKernelGGL(moe_reduce_kernel, dim3(E + 1), dim3(kMoeThreads), 0, st,
                     part_mass, part_count, part_tot, nb, E, (unsigned char*)stats);
  return hipGetLastError();
}

hipError_t launch_moe_loss(const void* stats, int E, int k, double coef, double* f, double* pe, double* loss,
                           hipStream_t st) {
  ProfileScope ps("moe_loss", st);
  hipLaunchKernelGGL(moe_loss_kernel, dim3(1), dim3(kMoeThreads), 0, st, (const unsigned char*)stats, E, k, coef,
                     f, pe, loss);
  return hipGetLastError();
}

hipError_t launch_moe_grad(const void* stats, int E, int k, double scale, int n, int mult, const int* mu,
                           float* dp, hipStream_t st) {
  const long threads = (long)n * (E / 4);
  if (threads == 0) return hipSuccess;
  ProfileScope ps("moe_grad", st);
  hipLaunchKernelGGL(moe_grad_kernel, dim3((unsigned)((threads + kMoeThreads - 1) / kMoeThreads)),
                     dim3(kMoeThreads), 0, st, (const unsigned char*)stats, E, k, scale, n, mult, mu, dp);
  return hipGetLastError();
}

}  // namespace spr
