// fp32 storage path: plain vector-ALU kernels, one thread per query row or
// per key.  On MI355X the fp32 matrix-core peak equals the fp32 vector peak
// (157.3 TFLOP/s), so fp32 gains nothing from MFMA; this path exists for
// full-precision parity and is fully deterministic (dQ comes from its own
// query-outer kernel, no atomics).
//
// Paper equations: forward H = softmax(S) V with the causal mask (App. A.1);
// backward dV = P^T dO, dP = dO V^T, dS = P * (dP - rowsum(dP * P)),
// dQ = dS K / sqrt(d), dK = dS^T Q / sqrt(d) (App. A.2-A.4), evaluated per
// segment tile so prefix and suffix keys are read in place.
#include "common.hpp"
#include "launch.hpp"

namespace spr {

namespace {

constexpr int kF32Threads = 64;

// Query-outer tile decode shared by the forward and the dQ kernel.
struct QTile {
  bool prefix;   // rows are prefix rows
  int lp0;       // first local row of the tile
  int seg_len;   // rows in the segment
  int row_base;  // memory row of local row 0 (suffix: cu[s])
  int seq;       // suffix index (suffix rows only)
};

__device__ __forceinline__ bool decode_qtile(const AttnArgs& a, int bq, QTile& t) {
  const int tile = gridDim.x - 1 - blockIdx.x;  // longest rows first
  t.seq = a.seq_base + blockIdx.z;
  if (tile < a.n_prefix_q_tiles) {
    t.prefix = true;
    t.lp0 = tile * bq;
    t.seg_len = a.P;
    t.row_base = 0;
  } else {
    t.prefix = false;
    t.lp0 = (tile - a.n_prefix_q_tiles) * bq;
    const SegRows sg = suffix_rows(a.cu, t.seq, a.total_len);
    t.row_base = sg.base;
    t.seg_len = sg.len;
  }
  return t.lp0 < t.seg_len;
}

template <int D>
__device__ __forceinline__ void load_rows_f32(float (*dst)[D], const float* src, int nrows_valid,
                                              int row_stride_elems, int nrows) {
  // cooperative: nrows x D floats, rows >= nrows_valid are zero
  for (int i = threadIdx.x; i < nrows * (D / 4); i += blockDim.x) {
    const int r = i / (D / 4), c = (i % (D / 4)) * 4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < nrows_valid) v = *(const float4*)(src + (size_t)r * row_stride_elems + c);
    dst[r][c] = v.x; dst[r][c + 1] = v.y; dst[r][c + 2] = v.z; dst[r][c + 3] = v.w;
  }
}

}  // namespace

// ---------------------------------------------------------------- forward
template <int D>
__global__ __launch_bounds__(kF32Threads) void fwd_f32_kernel(AttnArgs a) {
  constexpr int BQ = kF32Threads, BK = 32;
  __shared__ float Ks[BK][D];
  __shared__ float Vs[BK][D];
  QTile t;
  if (!decode_qtile(a, BQ, t)) return;
  const int h = blockIdx.y, hk = h / (a.hq / a.hkv);
  const int lp = t.lp0 + threadIdx.x;
  const bool valid = lp < t.seg_len;
  const float* q_base = (const float*)(t.prefix ? a.q_p : a.q_s);
  float q[D], o[D];
  const size_t qoff = ((size_t)(t.row_base + (valid ? lp : 0)) * a.hq + h) * D;
#pragma unroll
  for (int d = 0; d < D; ++d) { q[d] = valid ? q_base[qoff + d] : 0.f; o[d] = 0.f; }
  float m = -INFINITY, l = 0.f;
  const int last_row = min(t.lp0 + BQ, t.seg_len) - 1;  // highest local row of the tile

  for (int seg = 0; seg < 2; ++seg) {
    // seg 0: prefix keys; seg 1: the suffix's own keys (suffix rows only)
    if (seg == 1 && t.prefix) break;
    const bool causal = (seg == 0) == t.prefix;  // same-segment keys are causal
    const int nkeys = seg == 0 ? (t.prefix ? min(a.P, last_row + 1) : a.P) : last_row + 1;
    const float* kb = (const float*)(seg == 0 ? a.k_p : a.k_s);
    const float* vb = (const float*)(seg == 0 ? a.v_p : a.v_s);
    const int kbase = seg == 0 ? 0 : t.row_base;
    for (int k0 = 0; k0 < nkeys; k0 += BK) {
      const int nk = min(BK, nkeys - k0);
      __syncthreads();
      load_rows_f32<D>(Ks, kb + ((size_t)(kbase + k0) * a.hkv + hk) * D, nk, a.hkv * D, BK);
      load_rows_f32<D>(Vs, vb + ((size_t)(kbase + k0) * a.hkv + hk) * D, nk, a.hkv * D, BK);
      __syncthreads();
      float s[BK];
      float mt = -INFINITY;
#pragma unroll 4
      for (int j = 0; j < BK; ++j) {
        float acc = 0.f;
#pragma unroll
        for (int d = 0; d < D; ++d) acc = fmaf(q[d], Ks[j][d], acc);
        const bool vis = j < nk && (!causal || k0 + j <= lp);
        s[j] = vis ? acc * a.scale_log2 : -INFINITY;
        mt = fmaxf(mt, s[j]);
      }
      const float mn = fmaxf(m, mt);
      const float mu = mn == -INFINITY ? 0.f : mn;
      const float corr = exp2f(m - mu);
      l *= corr;
#pragma unroll
      for (int d = 0; d < D; ++d) o[d] *= corr;
#pragma unroll 4
      for (int j = 0; j < BK; ++j) {
        const float p = exp2f(s[j] - mu);
        l += p;
#pragma unroll
        for (int d = 0; d < D; ++d) o[d] = fmaf(p, Vs[j][d], o[d]);
      }
      m = mn;
    }
  }
  if (!valid) return;
  const float inv = 1.f / l;
  float* o_base = (float*)(t.prefix ? a.o_p : a.o_s);
#pragma unroll
  for (int d = 0; d < D; ++d) o_base[qoff + d] = o[d] * inv;
  float* lse = t.prefix ? a.lse_p : a.lse_s;
  lse[(size_t)(t.row_base + lp) * a.hq + h] = (m + log2f(l)) * kLn2;
}

// ------------------------------------------------------- backward, dK / dV
// Key-outer: one thread per key of a 64-key tile, looping over every query
// row that sees the tile (all G heads of the kv head).
template <int D>
__global__ __launch_bounds__(kF32Threads) void bwd_kv_f32_kernel(AttnArgs a) {
  constexpr int BK = kF32Threads, BQ = 16;
  __shared__ float Ks[BK][D + 1];
  __shared__ float Vs[BK][D + 1];
  __shared__ float Qs[BQ][D];
  __shared__ float dOs[BQ][D];
  __shared__ float Ls[BQ], Dd[BQ];
  const int x = blockIdx.x, hk = blockIdx.y, G = a.hq / a.hkv;
  bool kpre;
  int k0, kseg, kbase, s = 0;
  if (x < a.n_prefix_k_tiles) {
    kpre = true; k0 = x * BK; kseg = a.P; kbase = 0;
  } else {
    const int y = x - a.n_prefix_k_tiles;
    s = a.seq_base + y / a.n_suffix_k_tiles;
    k0 = (y % a.n_suffix_k_tiles) * BK;
    const SegRows sg = suffix_rows(a.cu, s, a.total_len);
    kbase = sg.base;
    kseg = sg.len;
    kpre = false;
  }
  if (k0 >= kseg) return;
  const int key = k0 + threadIdx.x;
  const bool kvalid = key < kseg;
  {
    const float* kb = (const float*)(kpre ? a.k_p : a.k_s);
    const float* vb = (const float*)(kpre ? a.v_p : a.v_s);
    const size_t off = ((size_t)(kbase + (kvalid ? key : 0)) * a.hkv + hk) * D;
    for (int d = 0; d < D; ++d) {
      Ks[threadIdx.x][d] = kvalid ? kb[off + d] : 0.f;
      Vs[threadIdx.x][d] = kvalid ? vb[off + d] : 0.f;
    }
  }
  float dk[D], dv[D];
#pragma unroll
  for (int d = 0; d < D; ++d) { dk[d] = 0.f; dv[d] = 0.f; }
  const float lse_scale = kLog2e;

  // row range job: rows [r0, r1) of a segment, memory row = base + r,
  // causal => row r sees key iff key <= r (same segment coordinates)
  auto run_rows = [&](int hh, bool rows_prefix, int base, int r0, int r1, bool causal) {
    const float* qb = (const float*)(rows_prefix ? a.q_p : a.q_s);
    const float* db = (const float*)(rows_prefix ? a.do_p : a.do_s);
    const float* lb = rows_prefix ? a.lse_p : a.lse_s;
    const float* ddb = rows_prefix ? a.dd_p : a.dd_s;
    for (int rt = r0; rt < r1; rt += BQ) {
      const int nr = min(BQ, r1 - rt);
      __syncthreads();
      load_rows_f32<D>(Qs, qb + ((size_t)(base + rt) * a.hq + hh) * D, nr, a.hq * D, BQ);
      load_rows_f32<D>(dOs, db + ((size_t)(base + rt) * a.hq + hh) * D, nr, a.hq * D, BQ);
      if (threadIdx.x < BQ) {
        const bool v = threadIdx.x < nr;
        Ls[threadIdx.x] = v ? lb[(size_t)(base + rt + threadIdx.x) * a.hq + hh] : 0.f;
        Dd[threadIdx.x] = v ? ddb[(size_t)(base + rt + threadIdx.x) * a.hq + hh] : 0.f;
      }
      __syncthreads();
      for (int r = 0; r < nr; ++r) {
        const bool vis = kvalid && (!causal || key <= rt + r);
        if (!vis) continue;
        float sc = 0.f, dp = 0.f;
#pragma unroll
        for (int d = 0; d < D; ++d) {
          sc = fmaf(Qs[r][d], Ks[threadIdx.x][d], sc);
          dp = fmaf(dOs[r][d], Vs[threadIdx.x][d], dp);
        }
        const float p = exp2f(sc * a.scale_log2 - Ls[r] * lse_scale);
        const float ds = p * (dp - Dd[r]);
#pragma unroll
        for (int d = 0; d < D; ++d) {
          dv[d] = fmaf(p, dOs[r][d], dv[d]);
          dk[d] = fmaf(ds, Qs[r][d], dk[d]);
        }
      }
    }
  };

  for (int hh = hk * G; hh < hk * G + G; ++hh) {
    if (kpre) {
      if (a.prefix_rows) run_rows(hh, true, 0, k0, a.P, true);
      if (a.suffix_rows) {
        const SegRows sp = suffix_span(a.cu, a.seq_base, a.seq_base + a.n_seq, a.total_len);
        const int r0 = sp.base, r1 = sp.base + sp.len;
        run_rows(hh, false, r0, 0, r1 - r0, false);
      }
    } else {
      run_rows(hh, false, kbase, k0, kseg, true);
    }
  }
  if (!kvalid) return;
  if (kpre) {
    const size_t off = ((size_t)key * a.hkv + hk) * D;
    if (a.pk_mode == kPkAccumulate) {
      for (int d = 0; d < D; ++d) {
        a.gk[off + d] += dk[d] * a.scale;
        a.gv[off + d] += dv[d];
      }
    } else {
      float* okp = (float*)a.dk_p;
      float* ovp = (float*)a.dv_p;
      for (int d = 0; d < D; ++d) {
        okp[off + d] = dk[d] * a.scale + a.gk[off + d];
        ovp[off + d] = dv[d] + a.gv[off + d];
      }
    }
  } else {
    const size_t off = ((size_t)(kbase + key) * a.hkv + hk) * D;
    float* oks = (float*)a.dk_s;
    float* ovs = (float*)a.dv_s;
    for (int d = 0; d < D; ++d) {
      oks[off + d] = dk[d] * a.scale;
      ovs[off + d] = dv[d];
    }
  }
}

// ------------------------------------------------------------ backward, dQ
// Query-outer: one thread per query row; dq_acc[row] += dS K (unscaled).
template <int D>
__global__ __launch_bounds__(kF32Threads) void bwd_q_f32_kernel(AttnArgs a) {
  constexpr int BQ = kF32Threads, BK = 32;
  __shared__ float Qs[BQ][D + 1];
  __shared__ float dOs[BQ][D + 1];
  __shared__ float Ks[BK][D];
  __shared__ float Vs[BK][D];
  QTile t;
  if (!decode_qtile(a, BQ, t)) return;
  const int h = blockIdx.y, hk = h / (a.hq / a.hkv);
  const int lp = t.lp0 + threadIdx.x;
  const bool valid = lp < t.seg_len;
  const float* qb = (const float*)(t.prefix ? a.q_p : a.q_s);
  const float* db = (const float*)(t.prefix ? a.do_p : a.do_s);
  const size_t qoff = ((size_t)(t.row_base + (valid ? lp : 0)) * a.hq + h) * D;
  for (int d = 0; d < D; ++d) {
    Qs[threadIdx.x][d] = valid ? qb[qoff + d] : 0.f;
    dOs[threadIdx.x][d] = valid ? db[qoff + d] : 0.f;
  }
  const size_t lidx = (size_t)(t.row_base + (valid ? lp : 0)) * a.hq + h;
  const float lse2 = valid ? (t.prefix ? a.lse_p : a.lse_s)[lidx] * kLog2e : 0.f;
  const float drow = valid ? (t.prefix ? a.dd_p : a.dd_s)[lidx] : 0.f;
  float dq[D];
#pragma unroll
  for (int d = 0; d < D; ++d) dq[d] = 0.f;
  const int last_row = min(t.lp0 + BQ, t.seg_len) - 1;
  for (int seg = 0; seg < 2; ++seg) {
    if (seg == 1 && t.prefix) break;
    const bool causal = (seg == 0) == t.prefix;
    const int nkeys = seg == 0 ? (t.prefix ? min(a.P, last_row + 1) : a.P) : last_row + 1;
    const float* kbp = (const float*)(seg == 0 ? a.k_p : a.k_s);
    const float* vbp = (const float*)(seg == 0 ? a.v_p : a.v_s);
    const int kbase = seg == 0 ? 0 : t.row_base;
    for (int k0 = 0; k0 < nkeys; k0 += BK) {
      const int nk = min(BK, nkeys - k0);
      __syncthreads();
      load_rows_f32<D>(Ks, kbp + ((size_t)(kbase + k0) * a.hkv + hk) * D, nk, a.hkv * D, BK);
      load_rows_f32<D>(Vs, vbp + ((size_t)(kbase + k0) * a.hkv + hk) * D, nk, a.hkv * D, BK);
      __syncthreads();
      if (!valid) continue;
      for (int j = 0; j < nk; ++j) {
        if (causal && k0 + j > lp) break;
        float sc = 0.f, dp = 0.f;
#pragma unroll
        for (int d = 0; d < D; ++d) {
          sc = fmaf(Qs[threadIdx.x][d], Ks[j][d], sc);
          dp = fmaf(dOs[threadIdx.x][d], Vs[j][d], dp);
        }
        const float ds = exp2f(sc * a.scale_log2 - lse2) * (dp - drow);
#pragma unroll
        for (int d = 0; d < D; ++d) dq[d] = fmaf(ds, Ks[j][d], dq[d]);
      }
    }
  }
  if (!valid) return;
  float* acc = t.prefix ? a.dq_acc_p : a.dq_acc_s;
  for (int d = 0; d < D; ++d) acc[qoff + d] += dq[d];
}

// ------------------------------------------------------------- launchers
int f32_block_q() { return kF32Threads; }
int f32_block_k() { return kF32Threads; }

hipError_t launch_fwd_f32(const AttnArgs& a, int head_dim, int n_z, hipStream_t st) {
  const dim3 grid(a.n_prefix_q_tiles + a.n_suffix_q_tiles, a.hq, n_z);
  if (grid.x == 0 || n_z == 0) return hipSuccess;
  ProfileScope ps("fwd_f32", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(fwd_f32_kernel<64>, grid, dim3(kF32Threads), 0, st, a);
  else
    hipLaunchKernelGGL(fwd_f32_kernel<128>, grid, dim3(kF32Threads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_bwd_f32(const AttnArgs& a, int head_dim, int n_qz, hipStream_t st) {
  {
    const dim3 grid(a.n_prefix_k_tiles + a.n_seq * a.n_suffix_k_tiles, a.hkv, 1);
    if (grid.x > 0) {
      ProfileScope ps("bwd_kv_f32", st);
      if (head_dim == 64)
        hipLaunchKernelGGL(bwd_kv_f32_kernel<64>, grid, dim3(kF32Threads), 0, st, a);
      else
        hipLaunchKernelGGL(bwd_kv_f32_kernel<128>, grid, dim3(kF32Threads), 0, st, a);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  const dim3 grid(a.n_prefix_q_tiles + a.n_suffix_q_tiles, a.hq, n_qz);
  if (grid.x == 0 || n_qz == 0) return hipSuccess;
  ProfileScope ps("bwd_q_f32", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(bwd_q_f32_kernel<64>, grid, dim3(kF32Threads), 0, st, a);
  else
    hipLaunchKernelGGL(bwd_q_f32_kernel<128>, grid, dim3(kF32Threads), 0, st, a);
  return hipGetLastError();
}

}  // namespace spr
