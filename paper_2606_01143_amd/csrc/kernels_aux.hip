// Bandwidth-bound helper kernels: the backward's row statistic
// D = rowsum(dO * O), fp32 accumulator conversion, zero fill, and the
// standalone gradient-cache accumulation G += g.
//
// All of them stream memory once with 16-byte vector accesses; the fill and
// accumulate kernels are grid-stride loops sized to a few waves per CU.
#include "common.hpp"

#include "launch.hpp"

namespace spr {

namespace {

constexpr int kAuxThreads = 256;

int aux_blocks(size_t n_vec) {
  size_t b = (n_vec + kAuxThreads - 1) / kAuxThreads;
  const size_t cap = 256 * 8;  // 8 workgroups per CU on 256 CUs
  if (b > cap) b = cap;
  if (b == 0) b = 1;
  return (int)b;
}

}  // namespace

// LPR lanes per (row, head), each loading 16 consecutive bytes of dO and of
// O, then a shuffle reduction over those lanes.  With cu != nullptr the rows
// are those of suffix `seq` only: cu[seq] .. cu[seq+1]-1 (clamped into the
// total_rows rows of the buffers), and `rows` is an upper bound on their
// count.  Also converts the row's LSE to the log2
// domain the backward kernels use: lse2 = lse * log2(e).
template <typename T, int D>
__global__ __launch_bounds__(kAuxThreads) void row_dot_kernel(const T* __restrict__ dO,
                                                            const T* __restrict__ O, int rows,
                                                            int total_rows,
                                                            const int32_t* __restrict__ cu,
                                                            int seq, int hq,
                                                            float* __restrict__ dd,
                                                            const float* __restrict__ lse,
                                                            float* __restrict__ lse2) {
  constexpr int VEC = 16 / (int)sizeof(T);  // elements per 16-byte load
  constexpr int LPR = D / VEC;              // lanes per (row, head): 8, 16 or 32
  const long tid = (long)blockIdx.x * kAuxThreads + threadIdx.x;
  const long item = tid / LPR;              // (row - row0) * hq + head
  const int sub = (int)(tid % LPR);
  int row0 = 0, nrows = rows;
  if (cu != nullptr) {
    const SegRows sg = suffix_rows(cu, seq, total_rows);
    row0 = sg.base;
    nrows = min(sg.len, rows);
  }
  // items past the end still take part in the shuffles (a group of LPR
  // lanes never straddles the end), but load and store nothing
  const bool valid = item < (long)nrows * hq;
  const size_t rh = (size_t)row0 * hq + (valid ? item : 0);
  float acc = 0.f;
  if (dO != nullptr && valid) {
    const size_t off = rh * D + (size_t)sub * VEC;
    if constexpr (sizeof(T) == 2) {
      const bf16x8 a = *(const bf16x8*)(dO + off);
      const bf16x8 b = *(const bf16x8*)(O + off);
#pragma unroll
      for (int k = 0; k < 8; ++k) acc += (float)a[k] * (float)b[k];
    } else {
      const float4 a = *(const float4*)(dO + off);
      const float4 b = *(const float4*)(O + off);
      acc = a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
    }
  }
#pragma unroll
  for (int m = LPR / 2; m >= 1; m >>= 1) acc += __shfl_xor(acc, m);
  if (valid && sub == 0) {
    dd[rh] = acc;
    lse2[rh] = lse[rh] * kLog2e;
  }
}

__global__ __launch_bounds__(kAuxThreads) void fill_zero_kernel(float4* p, size_t n4) {
  for (size_t i = (size_t)blockIdx.x * kAuxThreads + threadIdx.x; i < n4;
       i += (size_t)gridDim.x * kAuxThreads)
    p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

__global__ __launch_bounds__(kAuxThreads) void accumulate_kernel(float4* __restrict__ dst,
                                                                const float4* __restrict__ src,
                                                                size_t n4) {
  for (size_t i = (size_t)blockIdx.x * kAuxThreads + threadIdx.x; i < n4;
       i += (size_t)gridDim.x * kAuxThreads) {
    float4 a = dst[i];
    const float4 b = src[i];
    a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
    dst[i] = a;
  }
}

template <typename T>
__global__ __launch_bounds__(kAuxThreads) void convert_kernel(const float4* __restrict__ acc,
                                                             float scale,
                                                             const float4* __restrict__ add,
                                                             T* __restrict__ out, size_t n4) {
  for (size_t i = (size_t)blockIdx.x * kAuxThreads + threadIdx.x; i < n4;
       i += (size_t)gridDim.x * kAuxThreads) {
    float4 v = acc[i];
    v.x *= scale; v.y *= scale; v.z *= scale; v.w *= scale;
    if (add != nullptr) {
      const float4 b = add[i];
      v.x += b.x; v.y += b.y; v.z += b.z; v.w += b.w;
    }
    out[4 * i + 0] = from_f32<T>(v.x);
    out[4 * i + 1] = from_f32<T>(v.y);
    out[4 * i + 2] = from_f32<T>(v.z);
    out[4 * i + 3] = from_f32<T>(v.w);
  }
}

hipError_t launch_row_dot(int dtype, const void* dO, const void* O, int rows, int total_rows,
                          const int32_t* cu, int seq, int hq, int head_dim, float* dd,
                          const float* lse, float* lse2, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const size_t lpr = (size_t)head_dim * (dtype == 0 ? 4 : 2) / 16;  // lanes per (row, head)
  const size_t threads = (size_t)rows * hq * lpr;
  const int blocks = (int)((threads + kAuxThreads - 1) / kAuxThreads);
  ProfileScope ps("row_dot", st);
  if (dtype == 0) {
    if (head_dim == 64)
      hipLaunchKernelGGL((row_dot_kernel<float, 64>), blocks, kAuxThreads, 0, st,
                         (const float*)dO, (const float*)O, rows, total_rows, cu, seq, hq, dd, lse, lse2);
    else
      hipLaunchKernelGGL((row_dot_kernel<float, 128>), blocks, kAuxThreads, 0, st,
                         (const float*)dO, (const float*)O, rows, total_rows, cu, seq, hq, dd, lse, lse2);
  } else {
    if (head_dim == 64)
      hipLaunchKernelGGL((row_dot_kernel<bf16, 64>), blocks, kAuxThreads, 0, st,
                         (const bf16*)dO, (const bf16*)O, rows, total_rows, cu, seq, hq, dd, lse, lse2);
    else
      hipLaunchKernelGGL((row_dot_kernel<bf16, 128>), blocks, kAuxThreads, 0, st,
                         (const bf16*)dO, (const bf16*)O, rows, total_rows, cu, seq, hq, dd, lse, lse2);
  }
  return hipGetLastError();
}

hipError_t launch_fill_zero(float* p, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const size_t n4 = n / 4;  // every buffer here is a multiple of 4 floats
  ProfileScope ps("fill_zero", st);
  hipLaunchKernelGGL(fill_zero_kernel, aux_blocks(n4), kAuxThreads, 0, st, (float4*)p, n4);
  return hipGetLastError();
}

hipError_t launch_accumulate(float* dst, const float* src, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const size_t n4 = n / 4;
  ProfileScope ps("gkv_accumulate", st);
  hipLaunchKernelGGL(accumulate_kernel, aux_blocks(n4), kAuxThreads, 0, st, (float4*)dst,
                     (const float4*)src, n4);
  return hipGetLastError();
}

hipError_t launch_convert(int dtype, const float* acc, float scale, const float* add, void* out,
                          size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const size_t n4 = n / 4;
  ProfileScope ps("convert", st);
  if (dtype == 0)
    hipLaunchKernelGGL(convert_kernel<float>, aux_blocks(n4), kAuxThreads, 0, st,
                       (const float4*)acc, scale, (const float4*)add, (float*)out, n4);
  else
    hipLaunchKernelGGL(convert_kernel<bf16>, aux_blocks(n4), kAuxThreads, 0, st,
                       (const float4*)acc, scale, (const float4*)add, (bf16*)out, n4);
  return hipGetLastError();
}

// ------------------------------------------------- padded suffix layout
// Batch-plus-padding suffix tensors [n, s_max, row] are gathered into the
// packed layout [sum len, row] the attention kernels take, and the packed
// outputs scattered back (padding rows set to zero).

// cu[0..n] = exclusive prefix sum of the lengths clamped into [0, s_max]
// (clamped so that no gather or scatter can leave its buffers), lens_c the
// clamped lengths.  One block: the lengths go through LDS in chunks, one
// thread adds them in order.
__global__ __launch_bounds__(kAuxThreads) void seq_offsets_kernel(const int32_t* __restrict__ lens, int n,
                                                                  int s_max, int32_t* __restrict__ cu,
                                                                  int32_t* __restrict__ lens_c) {
  __shared__ int32_t chunk[kAuxThreads];
  int32_t run = 0;
  for (int base = 0; base < n; base += kAuxThreads) {
    const int i = base + (int)threadIdx.x;
    if (i < n) {
      const int32_t l = min(max(lens[i], 0), s_max);
      chunk[threadIdx.x] = l;
      lens_c[i] = l;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      const int m = min(kAuxThreads, n - base);
      for (int j = 0; j < m; ++j) {
        cu[base + j] = run;
        run += chunk[j];
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) cu[n] = run;
}

// Several tensors' rows in one launch.  Tensor j moves row_units[j] units
// of 16 bytes (wide[j]) or 4 bytes per row; thread idx takes one unit of one
// padded row.  Gather: packed[cu[i] + t] = padded[i, t] for t < lens_c[i].
// Scatter: padded[i, t] = packed[cu[i] + t], or zero for padding rows.
struct RowMoves {
  const void* src[kMaxRowMoves];
  void* dst[kMaxRowMoves];
  int units[kMaxRowMoves];
  int wide[kMaxRowMoves];
  int count, units_per_row;
};

// With few suffixes (n <= kLdsSeqs) each block derives the offsets itself
// from the raw lengths (clamped as in seq_offsets_kernel), and block 0 of a
// gather also stores them to cu_pre / lens_pre for the packed kernels that
// follow, so no separate offsets launch is needed; otherwise cu / lens_c
// come precomputed.
constexpr int kLdsSeqs = 1024;
__global__ __launch_bounds__(kAuxThreads) void rows_move_kernel(RowMoves m, const int32_t* __restrict__ lens,
                                                                int n, const int32_t* __restrict__ cu_pre,
                                                                const int32_t* __restrict__ lens_pre, int s_max,
                                                                long total, int gather) {
  __shared__ int32_t cu_s[kLdsSeqs + 1], len_s[kLdsSeqs];
  const int32_t *cu = cu_pre, *lens_c = lens_pre;
  if (lens != nullptr) {
    for (int i = threadIdx.x; i < n; i += kAuxThreads) len_s[i] = min(max(lens[i], 0), s_max);
    __syncthreads();
    if (threadIdx.x == 0) {
      int32_t run = 0;
      for (int i = 0; i < n; ++i) {
        cu_s[i] = run;
        run += len_s[i];
      }
      cu_s[n] = run;
    }
    __syncthreads();
    cu = cu_s;
    lens_c = len_s;
    if (gather && blockIdx.x == 0) {
      int32_t* cu_out = const_cast<int32_t*>(cu_pre);
      int32_t* len_out = const_cast<int32_t*>(lens_pre);
      for (int i = threadIdx.x; i <= n; i += kAuxThreads) cu_out[i] = cu_s[i];
      for (int i = threadIdx.x; i < n; i += kAuxThreads) len_out[i] = len_s[i];
    }
  }
  const long idx = (long)blockIdx.x * kAuxThreads + threadIdx.x;
  if (idx >= total) return;
  const long pr = idx / m.units_per_row;
  int u = (int)(idx % m.units_per_row);
  int j = 0;
  while (u >= m.units[j]) {
    u -= m.units[j];
    ++j;
  }
  const int i = (int)(pr / s_max), t = (int)(pr % s_max);
  const bool valid = t < lens_c[i];
  const long prow = valid ? (long)cu[i] + t : 0;
  const long pad_off = pr * m.units[j] + u, pack_off = prow * m.units[j] + u;
  if (m.wide[j]) {
    if (gather) {
      if (valid) ((float4*)m.dst[j])[pack_off] = ((const float4*)m.src[j])[pad_off];
    } else {
      ((float4*)m.dst[j])[pad_off] = valid ? ((const float4*)m.src[j])[pack_off] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  } else {
    if (gather) {
      if (valid) ((float*)m.dst[j])[pack_off] = ((const float*)m.src[j])[pad_off];
    } else {
      ((float*)m.dst[j])[pad_off] = valid ? ((const float*)m.src[j])[pack_off] : 0.f;
    }
  }
}

hipError_t launch_seq_offsets(const int32_t* lens, int n, int s_max, int32_t* cu, int32_t* lens_c,
                              hipStream_t st) {
  ProfileScope ps("seq_offsets", st);
  hipLaunchKernelGGL(seq_offsets_kernel, dim3(1), dim3(kAuxThreads), 0, st, lens, n, s_max, cu, lens_c);
  return hipGetLastError();
}

bool rows_move_needs_offsets(int n) { return n > kLdsSeqs; }

hipError_t launch_rows_move(bool gather, const RowMove* moves, int count, const int32_t* lens, const int32_t* cu,
                            const int32_t* lens_c, int n, int s_max, hipStream_t st) {
  if (count < 1 || count > kMaxRowMoves) return hipErrorInvalidValue;
  RowMoves m;
  m.count = count;
  m.units_per_row = 0;
  for (int j = 0; j < count; ++j) {
    const RowMove& x = moves[j];
    // 16-byte units when rows and pointers allow, else 4-byte units
    const bool wide = x.row_bytes % 16 == 0 && ((uintptr_t)x.src & 15) == 0 && ((uintptr_t)x.dst & 15) == 0;
    m.src[j] = x.src;
    m.dst[j] = x.dst;
    m.wide[j] = wide ? 1 : 0;
    m.units[j] = (int)(x.row_bytes / (wide ? 16 : 4));
    m.units_per_row += m.units[j];
  }
  for (int j = count; j < kMaxRowMoves; ++j) {
    m.src[j] = nullptr;
    m.dst[j] = nullptr;
    m.units[j] = 0;
    m.wide[j] = 0;
  }
  const long total = (long)n * s_max * m.units_per_row;
  if (total == 0) return hipSuccess;
  const unsigned nb = (unsigned)((total + kAuxThreads - 1) / kAuxThreads);
  ProfileScope ps(gather ? "rows_gather" : "rows_scatter", st);
  hipLaunchKernelGGL(rows_move_kernel, dim3(nb), dim3(kAuxThreads), 0, st, m, n <= kLdsSeqs ? lens : nullptr, n,
                     cu, lens_c, s_max, total, gather ? 1 : 0);
  return hipGetLastError();
}

}  // namespace spr
