// bf16 forward attention on gfx950 matrix cores (Phase A prefix forward,
// Phase B suffix forward, and the dense baseline's forward).
//
// What it computes (paper Sec. 3.1 and App. A.1): for each query row,
// O = softmax(S) V over the row's visible keys, S = scale * q k^T, with one
// joint softmax across the prefix keys and the row's own causal suffix keys
// (H_2 = P_21 V_1 + P_22 V_2), plus the row's natural-log LSE.
//
// Structure: one workgroup = 4 waves = 128 query rows of one q head (or, in
// the twelve-wave form of large unsplit launches, 12 waves = 96 rows of the
// four q heads of one kv head); each wave owns 32 rows of one head.  Keys
// stream through LDS in 64-row tiles, first the prefix tiles (read in place
// from K_P/V_P), then the suffix's own tiles.
// Tiles are double-buffered: the next tile's direct-to-LDS loads are issued
// before the current tile's products.  Per tile and wave
// (v_mfma_f32_32x32x16_bf16, operand conventions in tile.hpp):
//   S^T (64 keys x 32 rows) = K Q^T   A = K tile rows, B = Q (registers)
//   O^T (d x 32 rows)      += V^T P^T  A = V tile read transposed,
//                                      B = P^T straight from the S^T registers
// With S^T each lane holds 16 keys of ONE query row, so the online softmax
// needs a single cross-lane exchange per statistic.
#include <algorithm>

#include "common.hpp"
#include "launch.hpp"
#include "tile.hpp"

namespace spr {

namespace {
constexpr int kFwdBQ = 128;
constexpr int kFwdWideBQ = 96;  // rows of the twelve-wave prefix launch (per q head)
// headroom (log2 domain) of the softmax reference over a row's true running
// max: P = exp2(s - m) stays below 256, far inside fp32, and bf16 rounds it
// to the same relative precision as below 1
constexpr float kFwdSlack = 8.f;
}  // namespace

int fwd_bf16_block_q() { return kFwdBQ; }

// Query-outer grids are 1D: block b -> (kv head b % Hkv, q head of that kv
// group, row tile, suffix).  Workgroups are dispatched round-robin over the
// eight XCDs, so every block of one kv head lands on the same XCD (for
// Hkv dividing 8) and the K/V it streams stays in that XCD's L2.
struct RowBlock {
  int tile, z, hq, split;
};
__device__ __forceinline__ RowBlock decode_row_block(const AttnArgs& a, int ntx) {
  const int G = a.hq / a.hkv;
  int b = blockIdx.x;
  const int hk = b % a.hkv;
  b /= a.hkv;
  const int gi = b % G;
  b /= G;
  RowBlock rb;
  rb.split = b % a.n_split;
  b /= a.n_split;
  rb.tile = ntx - 1 - b % ntx;  // rows with the most keys first
  rb.z = b / ntx;
  rb.hq = hk * G + gi;
  return rb;
}

// The forward in one of two workgroup forms.  Four waves: 128 rows of one q
// head, key splits allowed.  Twelve waves (WIDE, launches whose workgroups
// fill the GPU several times over): 96 rows of four q heads of one kv head,
// wave w on rows 32 (w / 4) .. + 31 of head w % 4, all twelve reading each
// K/V tile that waves 0-3 load, no key splits.  Both keep the 64 KB of
// double-buffered tiles, so only the twelve-wave form holds three waves on
// every SIMD, which needs the loop to fit in 168 registers.
template <int D, bool WIDE>
__device__ __forceinline__ void fwd_body(const AttnArgs& a, bf16 (&Ks)[2][Tile<D>::ELEMS],
                                         bf16 (&Vs)[2][Tile<D>::ELEMS]) {
  constexpr int NS = D / 16;   // k-steps over d for S^T
  constexpr int NDB = D / 32;  // 32-wide d blocks of O^T
  constexpr int BK = kTileRows;
  constexpr int BQ = WIDE ? kFwdWideBQ : kFwdBQ;

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int r = lane & 31, h = lane >> 5;
  FragOffsets<D> fo;
  fo.init(lane);

  // ---- which BQ query rows: prefix rows, or rows of suffix seq_base + z
  const int ntx = a.n_prefix_q_tiles + a.n_suffix_q_tiles;
  int hq, hk;
  RowBlock blk;
  if constexpr (WIDE) {
    // block b -> (kv head b % Hkv, group of four q heads, 96-row tile,
    // suffix), the rows with the most keys first
    const int G = a.hq / a.hkv;
    int b = blockIdx.x;
    hk = b % a.hkv;
    b /= a.hkv;
    const int hg = b % (G / 4);
    b /= G / 4;
    blk.tile = ntx - 1 - b % ntx;
    blk.z = b / ntx;
    blk.split = 0;
    hq = hk * G + 4 * hg + (w & 3);
  } else {
    blk = decode_row_block(a, ntx);
    hq = blk.hq;
    hk = hq / (a.hq / a.hkv);
  }
  const int seq = a.seq_base + blk.z;
  bool prefix_rows;
  int lp0, seg_len, row_base;
  if (blk.tile < a.n_prefix_q_tiles) {
    prefix_rows = true;
    lp0 = blk.tile * BQ;
    seg_len = a.P;
    row_base = 0;
  } else {
    prefix_rows = false;
    lp0 = (blk.tile - a.n_prefix_q_tiles) * BQ;
    const SegRows sg = suffix_rows(a.cu, seq, a.total_len);
    row_base = sg.base;
    seg_len = sg.len;
  }
  if (lp0 >= seg_len) return;
  const int wave_lp0 = lp0 + 32 * (WIDE ? w >> 2 : w);  // first row of this wave
  const int row_lp = wave_lp0 + r;    // this lane's query row (segment-local)
  const bool row_valid = row_lp < seg_len;
  const int my_lp = row_valid ? row_lp : seg_len - 1;  // rows past the end recompute the last one

  // Q as the B operand of S^T = K Q^T: slot (h, j) of k-step s is d = 16 s + 8 h + j
  bf16x8 qf[NS];
  {
    const bf16* qb = (const bf16*)(prefix_rows ? a.q_p : a.q_s);
    const size_t off = ((size_t)(row_base + my_lp) * a.hq + hq) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[s] = *(const bf16x8*)(qb + off + 16 * s);
#pragma unroll
    for (int s = 0; s < NS; ++s) settle(qf[s]);
  }
  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = zero16();
  float m = -INFINITY, l = 0.f;  // running max (log2 domain) and sum of row my_lp

  // key tiles: prefix keys first (causal for prefix rows), then own suffix keys
  const int last_lp = min(lp0 + BQ, seg_len) - 1;
  const int nkeys0 = prefix_rows ? min(a.P, last_lp + 1) : a.P;
  const int nkeys1 = prefix_rows ? 0 : last_lp + 1;
  const int nt0 = (nkeys0 + BK - 1) / BK, nt1 = (nkeys1 + BK - 1) / BK;
  // this block's contiguous share of the key tiles
  const int t_begin = (int)((long)(nt0 + nt1) * blk.split / a.n_split);
  const int t_end = (int)((long)(nt0 + nt1) * (blk.split + 1) / a.n_split);

  const bf16 *k_p = in_sgpr((const bf16*)a.k_p), *k_s = in_sgpr((const bf16*)a.k_s);
  const bf16 *v_p = in_sgpr((const bf16*)a.v_p), *v_s = in_sgpr((const bf16*)a.v_s);
  TileLoader<D, 4, BK> tl;
  tl.init(a.hkv, w & 3, lane);
  auto issue = [&](int t, bf16* Kd, bf16* Vd) {
    if (WIDE && w >= 4) return;  // waves 0-3 load every tile
    const int seg = t < nt0 ? 0 : 1;
    const int k0 = (seg == 0 ? t : t - nt0) * BK;
    const int nk = min(BK, (seg == 0 ? nkeys0 : nkeys1) - k0);
    const int kbase = seg == 0 ? 0 : row_base;
    tl.load(Kd, pick(seg == 0, k_p, k_s), kbase + k0, nk, a.hkv, hk);
    tl.load(Vd, pick(seg == 0, v_p, v_s), kbase + k0, nk, a.hkv, hk);
  };

  auto compute = [&](int t, const bf16* Kc, const bf16* Vc) {
    const int seg = t < nt0 ? 0 : 1;
    const int k0 = (seg == 0 ? t : t - nt0) * BK;
    const int nk = min(BK, (seg == 0 ? nkeys0 : nkeys1) - k0);
    const bool causal = (seg == 0) == prefix_rows;  // keys of the row's own segment
    if (causal && k0 > wave_lp0 + 31) return;       // no row of this wave sees the tile
    // S^T = K Q^T ; st[kb][i] = S^T[key k0 + 32 kb + c_row0(i) + 4 h][row my_lp]
    f32x16 st[2] = {zero16(), zero16()};
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) st[kb] = mfma32(row_frag<D>(Kc, fo, 32 * kb, s), qf[s], st[kb]);
    sched_reads_ahead<2 * NS, 1, 4>();
#define SC(e) st[(e) >> 4][(e) & 15]
    if (nk < BK || (causal && k0 + BK - 1 > wave_lp0)) {  // partial or diagonal tile
      // keys kk = 32 (e / 16) + c_row0(e % 16) + 4 h are visible iff kk < lim
      int lp = my_lp;  // recomputed in the twelve-wave form (registers)
      if constexpr (WIDE)
        lp = min(wave_lp0 + (int)(__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)) & 31),
                 seg_len - 1);
      const int lim = (causal ? min(nk, lp - k0 + 1) : nk) - 4 * h;
#pragma unroll
      for (int e = 0; e < 32; ++e) SC(e) = 32 * (e >> 4) + c_row0(e & 15) < lim ? SC(e) : -INFINITY;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int e = 0; e < 32; ++e) mt = fmaxf(mt, SC(e));
    mt = fmaxf(mt, __shfl_xor(mt, 32)) * a.scale_log2;
    // m is the reference the exponents are taken against, not necessarily
    // the running max: it moves (and O, l are rescaled) only when some row's
    // max exceeds it by more than kFwdSlack, so P = exp2(s - m) < 2^kFwdSlack.
    // O / l and m + log2(l) do not depend on the reference.
    if (__builtin_expect(__any(mt > m + kFwdSlack), 0)) {
      const float mn = fmaxf(m, mt);
      const float corr = fast_exp2(m - (mn == -INFINITY ? 0.f : mn));
      l *= corr;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] *= corr;
      m = mn;
    }
    const float mu = m == -INFINITY ? 0.f : m;
    float rs = 0.f;
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      SC(e) = fast_exp2(fmaf(SC(e), a.scale_log2, -mu));
      rs += SC(e);
    }
#undef SC
    rs += __shfl_xor(rs, 32);
    l += rs;
    // O^T += V^T P^T over 16-key steps u (C-order keys 16 u + k(h, j))
#pragma unroll
    for (int u = 0; u < BK / 16; ++u) {
      const bf16x8 pb = c_kfrag(st[u >> 1], u & 1);
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] = mfma32(tr_frag<D>(Vc, fo, 16 * u, db), pb, o[db]);
    }
    sched_reads_ahead<BK / 16 * NDB, 2, WIDE ? 1 : 2>();
  };

  if (t_begin < t_end) issue(t_begin, Ks[0], Vs[0]);
  tile_barrier();
  // two tiles per pass, so each buffer's LDS address is a constant and goes
  // into the reads' immediate offsets instead of a per-read address add
  for (int t = t_begin; t < t_end; t += 2) {
    if (t + 1 < t_end) issue(t + 1, Ks[1], Vs[1]);
    compiler_fence();
    compute(t, Ks[0], Vs[0]);
    tile_barrier();
    if (t + 1 >= t_end) break;
    if (t + 2 < t_end) issue(t + 2, Ks[0], Vs[0]);
    compiler_fence();
    compute(t + 1, Ks[1], Vs[1]);
    tile_barrier();
  }

  // (the twelve-wave form recomputes the lane and its row here: at 168
  // registers, values kept from before the loop would spill)
  int e_lp = my_lp, e_h = h;
  bool e_valid = row_valid;
  if constexpr (WIDE) {
    const int e_lane = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
    e_h = e_lane >> 5;
    e_lp = wave_lp0 + (e_lane & 31);
    e_valid = e_lp < seg_len;
  }
  if (!e_valid) return;
  if (!WIDE && a.n_split > 1) {
    // partial result of this key range: O / l and log2(sum) + max (a range
    // with no visible key gives l = 0: weight 0 in the combine)
    const size_t prow = ((size_t)blk.split * a.total_len + row_base + my_lp) * a.hq + hq;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    float* po = a.part_o + prow * D + 4 * h;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        *(float4*)(po + 32 * db + 8 * g4) = make_float4(o[db][4 * g4] * inv, o[db][4 * g4 + 1] * inv,
                                                        o[db][4 * g4 + 2] * inv, o[db][4 * g4 + 3] * inv);
    if (h == 0) a.part_lse[prow] = l > 0.f ? m + log2f(l) : -INFINITY;
    return;
  }
  // o[db][i] = O^T[d = 32 db + c_row0(i) + 4 h][row my_lp]
  const float inv = 1.f / l;
  bf16* ob = (bf16*)(prefix_rows ? a.o_p : a.o_s);
  const size_t off = ((size_t)(row_base + e_lp) * a.hq + hq) * D + 4 * e_h;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const bf16x4 v = {(bf16)(o[db][4 * g4] * inv), (bf16)(o[db][4 * g4 + 1] * inv),
                        (bf16)(o[db][4 * g4 + 2] * inv), (bf16)(o[db][4 * g4 + 3] * inv)};
      *(bf16x4*)(ob + off + 32 * db + 8 * g4) = v;
    }
  if (e_h == 0) {
    float* lse = prefix_rows ? a.lse_p : a.lse_s;
    lse[(size_t)(row_base + e_lp) * a.hq + hq] = (m + log2f(l)) * kLn2;
  }
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void fwd_bf16_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) bf16 Ks[2][Tile<D>::ELEMS];
  __shared__ __attribute__((aligned(1024))) bf16 Vs[2][Tile<D>::ELEMS];
  fwd_body<D, false>(a, Ks, Vs);
}

template <int D>
__global__ __launch_bounds__(3 * kThreads, 1) void fwd_wide_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) bf16 Ks[2][Tile<D>::ELEMS];
  __shared__ __attribute__((aligned(1024))) bf16 Vs[2][Tile<D>::ELEMS];
  fwd_body<D, true>(a, Ks, Vs);
}

// Merge of the n_split partial outputs of every (suffix row, q head):
// lse = log2 sum_j 2^lse_j, O = sum_j 2^(lse_j - lse) O_j.  One group of
// D / 4 threads per (row, head), 16-byte accesses.
template <int D>
__global__ __launch_bounds__(256) void fwd_combine_kernel(AttnArgs a) {
  constexpr int TPR = D / 4;  // threads per (row, head)
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const long rh = idx / TPR;  // row * hq + head
  const int c = (int)(idx % TPR);
  const long nrh = (long)a.total_len * a.hq;
  if (rh >= nrh) return;
  float mx = -INFINITY;
  for (int j = 0; j < a.n_split; ++j) mx = fmaxf(mx, a.part_lse[(size_t)j * nrh + rh]);
  float sum = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < a.n_split; ++j) {
    const float lj = a.part_lse[(size_t)j * nrh + rh];
    const float wj = lj == -INFINITY ? 0.f : exp2f(lj - mx);
    const float4 oj = *(const float4*)(a.part_o + ((size_t)j * nrh + rh) * D + 4 * c);
    sum += wj;
    acc.x += wj * oj.x;
    acc.y += wj * oj.y;
    acc.z += wj * oj.z;
    acc.w += wj * oj.w;
  }
  const float inv = 1.f / sum;
  const bf16x4 v = {(bf16)(acc.x * inv), (bf16)(acc.y * inv), (bf16)(acc.z * inv), (bf16)(acc.w * inv)};
  *(bf16x4*)((bf16*)a.o_s + (size_t)rh * D + 4 * c) = v;
  if (c == 0) a.lse_s[rh] = (mx + log2f(sum)) * kLn2;
}

hipError_t launch_fwd_bf16(const AttnArgs& a, int head_dim, int n_z, hipStream_t st) {
  const long nb = (long)(a.n_prefix_q_tiles + a.n_suffix_q_tiles) * a.hq * n_z * a.n_split;
  if (nb == 0) return hipSuccess;
  ProfileScope ps("fwd_bf16", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(fwd_bf16_kernel<64>, dim3((unsigned)nb), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(fwd_bf16_kernel<128>, dim3((unsigned)nb), dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_split <= 1) return e;
  const long threads = (long)a.total_len * a.hq * (head_dim / 4);
  const unsigned cb = (unsigned)((threads + 255) / 256);
  ProfileScope pc("fwd_combine", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(fwd_combine_kernel<64>, dim3(cb), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(fwd_combine_kernel<128>, dim3(cb), dim3(256), 0, st, a);
  return hipGetLastError();
}

// The forward in its twelve-wave form: a.n_prefix_q_tiles and
// a.n_suffix_q_tiles count 96-row tiles; no key splits, four q heads per kv
// head or a multiple of four.
hipError_t launch_fwd_bf16_wide(const AttnArgs& a, int head_dim, int n_z, hipStream_t st) {
  const int G = a.hq / a.hkv;
  if (G % 4 != 0 || a.n_split > 1) return hipErrorInvalidValue;
  const long nb = (long)(a.n_prefix_q_tiles + a.n_suffix_q_tiles) * n_z * a.hkv * (G / 4);
  if (nb == 0) return hipSuccess;
  ProfileScope ps("fwd_bf16", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(fwd_wide_kernel<64>, dim3((unsigned)nb), dim3(3 * kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(fwd_wide_kernel<128>, dim3((unsigned)nb), dim3(3 * kThreads), 0, st, a);
  return hipGetLastError();
}

int fwd_bf16_wide_block_q() { return kFwdWideBQ; }

int fwd_bf16_split(int n_row_blocks, int prefix_len) {
  // enough workgroups for two per CU on 256 CUs, each split keeping at
  // least four 64-key tiles of the prefix
  if (n_row_blocks <= 0) return 1;
  int ns = (512 + n_row_blocks - 1) / n_row_blocks;
  ns = std::min(ns, std::max(1, prefix_len / (4 * kTileRows)));
  return std::max(1, std::min(ns, 16));
}

}  // namespace spr
