// bf16 forward attention on gfx950 matrix cores (Phase A prefix forward,
// Phase B suffix forward, and the dense baseline's forward).
//
// What it computes (paper Sec. 3.1 and App. A.1): for each query row,
// O = softmax(S) V over the row's visible keys, S = scale * q k^T, with one
// joint softmax across the prefix keys and the row's own causal suffix keys
// (H_2 = P_21 V_1 + P_22 V_2), plus the row's natural-log LSE.
//
// Structure: one workgroup = 4 waves = 128 query rows of one q head; each
// wave owns 32 rows.  Keys stream through LDS in tiles of 64, first the
// prefix tiles (read in place from K_P/V_P), then the suffix's own tiles,
// double-buffered: the next tile's global loads are in flight while the
// current one is multiplied.  An online softmax carries the row max and
// sum across tiles.  Per tile and wave (v_mfma_f32_32x32x16_bf16):
//   S^T (64 keys x 32 rows) = K Q^T   A = K rows (natural tile), B = Q (registers)
//   O^T (d x 32 rows)      += V^T P^T  A = V columns (transposed tile),
//                                      B = P^T straight from the S^T registers
// Computing S^T leaves each lane holding 16 keys of one query row: the row
// max/sum need one cross-lane exchange, and the keys already sit in the
// B-operand slots of the PV product.
#include "common.hpp"
#include "launch.hpp"
#include "tile.hpp"

namespace spr {

namespace {
constexpr int kFwdBQ = 128;
constexpr int kFwdBK = 64;
constexpr int kFwdThreads = 256;
}  // namespace

int fwd_bf16_block_q() { return kFwdBQ; }

template <int D>
__global__ __launch_bounds__(kFwdThreads) void fwd_bf16_kernel(AttnArgs a) {
  using TG = TileGeom<D>;
  constexpr int BQ = kFwdBQ, BK = kFwdBK;
  constexpr int NS = D / 16;   // k-steps over d for S^T
  constexpr int NDB = D / 32;  // 32-wide d blocks of O^T
  __shared__ __attribute__((aligned(16))) bf16 Kn[2 * TG::NAT];
  __shared__ __attribute__((aligned(16))) bf16 Vt[2 * TG::TRN];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r = lane & 31, h = lane >> 5;

  // ---- which 128 query rows: prefix rows, or rows of suffix seq_base + z
  const int tile = gridDim.x - 1 - blockIdx.x;  // rows with the most keys first
  const int seq = a.seq_base + blockIdx.z;
  bool prefix_rows;
  int lp0, seg_len, row_base;
  if (tile < a.n_prefix_q_tiles) {
    prefix_rows = true;
    lp0 = tile * BQ;
    seg_len = a.P;
    row_base = 0;
  } else {
    prefix_rows = false;
    lp0 = (tile - a.n_prefix_q_tiles) * BQ;
    row_base = a.cu[seq];
    seg_len = a.cu[seq + 1] - row_base;
  }
  if (lp0 >= seg_len) return;
  const int hq = blockIdx.y, hk = hq / (a.hq / a.hkv);
  const int wave_lp0 = lp0 + 32 * w;  // first row of this wave
  const int my_lp = wave_lp0 + r;     // this lane's query row (segment-local)
  const bool row_valid = my_lp < seg_len;

  // Q as the B operand of S^T = K Q^T: slot (h, j) of k-step s is d = 16 s + 8 h + j
  bf16x8 qf[NS];
  {
    const bf16* qb = (const bf16*)(prefix_rows ? a.q_p : a.q_s);
    const size_t off = ((size_t)(row_base + (row_valid ? my_lp : 0)) * a.hq + hq) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[s] = row_valid ? *(const bf16x8*)(qb + off + 16 * s) : zero_bf8();
  }
  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = zero16();
  float m = -INFINITY, l = 0.f;  // running max (log2 domain) and sum of row my_lp

  // LDS offsets of this lane's fragments: K rows at k_off + immediates; the
  // V column of d block db is v_col + db * 32 * kTileRows, its 16-key step u
  // at chunk (2 u + h) ^ trn_swz(32 db + r)
  const int k_off = nat_off<D>(r, 0, h);
  const int v_col = r * kTileRows;

  // key tiles: prefix keys first (causal for prefix rows), then own suffix keys
  const int last_lp = min(lp0 + BQ, seg_len) - 1;
  const int nkeys0 = prefix_rows ? min(a.P, last_lp + 1) : a.P;
  const int nkeys1 = prefix_rows ? 0 : last_lp + 1;
  const int nt0 = (nkeys0 + BK - 1) / BK, nt1 = (nkeys1 + BK - 1) / BK;
  const int ntiles = nt0 + nt1;
  auto tile_info = [&](int t, int& seg, int& k0, int& nk) {
    seg = t < nt0 ? 0 : 1;
    k0 = (seg == 0 ? t : t - nt0) * BK;
    nk = min(BK, (seg == 0 ? nkeys0 : nkeys1) - k0);
  };
  Stager<D> sk, sv;
  auto stage_load = [&](int t) {
    int seg, k0, nk;
    tile_info(t, seg, k0, nk);
    const bf16* kb = (const bf16*)(seg == 0 ? a.k_p : a.k_s);
    const bf16* vb = (const bf16*)(seg == 0 ? a.v_p : a.v_s);
    const int kbase = seg == 0 ? 0 : row_base;
    sk.load(kb, kbase + k0, nk, a.hkv, hk, tid);
    sv.load(vb, kbase + k0, nk, a.hkv, hk, tid);
  };
  if (ntiles > 0) {
    stage_load(0);
    sk.store_nat(Kn, tid);
    sv.store_trn(Vt, tid);
  }
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) stage_load(t + 1);  // global loads in flight during the MFMAs
    int seg, k0, nk;
    tile_info(t, seg, k0, nk);
    const bool causal = (seg == 0) == prefix_rows;  // keys of the row's own segment
    if (!(causal && k0 > wave_lp0 + 31)) {          // else no row of this wave sees the tile
      const bf16* Kb = Kn + buf * TG::NAT + k_off;
      const bf16* Vb = Vt + buf * TG::TRN;
      // S^T = K Q^T ; st[kb][i] = S^T[key k0 + 32 kb + c_row(i, h)][row my_lp]
      f32x16 st[BK / 32];
#pragma unroll
      for (int kb = 0; kb < BK / 32; ++kb) st[kb] = zero16();
#pragma unroll
      for (int s = 0; s < NS; ++s)  // independent chains interleaved
#pragma unroll
        for (int kb = 0; kb < BK / 32; ++kb)
          st[kb] = mfma32(lds8(Kb, nat_off<D>(32 * kb, 16 * s, 0)), qf[s], st[kb]);
#define SC(e) st[(e) >> 4][(e) & 15]
      if (nk < BK || (causal && k0 + BK - 1 > wave_lp0)) {  // partial or diagonal tile
        const int lim = causal ? min(nk, my_lp - k0 + 1) : nk;  // keys kk < lim are visible
#pragma unroll
        for (int e = 0; e < BK / 2; ++e) SC(e) = 32 * (e >> 4) + c_row(e & 15, h) < lim ? SC(e) : -INFINITY;
      }
      float mt = -INFINITY;
#pragma unroll
      for (int e = 0; e < BK / 2; ++e) mt = fmaxf(mt, SC(e));
      mt = fmaxf(mt, __shfl_xor(mt, 32)) * a.scale_log2;
      const float mn = fmaxf(m, mt);
      const float mu = mn == -INFINITY ? 0.f : mn;
      if (__builtin_expect(__any(mn > m), 0)) {  // rescale only when some row's max grew
        const float corr = fast_exp2(m - mu);
        l *= corr;
#pragma unroll
        for (int db = 0; db < NDB; ++db) o[db] *= corr;
      }
      m = mn;
      float rs = 0.f;
#pragma unroll
      for (int e = 0; e < BK / 2; ++e) {
        SC(e) = fast_exp2(fmaf(SC(e), a.scale_log2, -mu));
        rs += SC(e);
      }
      rs += __shfl_xor(rs, 32);
      l += rs;
#undef SC
      // O^T += V^T P^T over 16-key steps u: keys 16 u + 8 h + 0..7
#pragma unroll
      for (int u = 0; u < BK / 16; ++u) {
        const bf16x8 pb = c_to_kfrag(st[u >> 1], u & 1);
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          o[db] = mfma32(lds8(Vb, v_col + db * 32 * kTileRows +
                                      8 * ((2 * u + h) ^ trn_swz(32 * db + r))),
                         pb, o[db]);
      }
    }
    compiler_fence();
    if (t + 1 < ntiles) {
      sk.store_nat(Kn + (buf ^ 1) * TG::NAT, tid);
      sv.store_trn(Vt + (buf ^ 1) * TG::TRN, tid);
    }
    __syncthreads();
  }

  if (!row_valid) return;
  // o[db][i] = O^T[d = 32 db + 8 (i/4) + 4 h + i%4][row my_lp]
  const float inv = 1.f / l;
  bf16* ob = (bf16*)(prefix_rows ? a.o_p : a.o_s);
  const size_t off = ((size_t)(row_base + my_lp) * a.hq + hq) * D + 4 * h;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const bf16x4 v = {(bf16)(o[db][4 * g4] * inv), (bf16)(o[db][4 * g4 + 1] * inv),
                        (bf16)(o[db][4 * g4 + 2] * inv), (bf16)(o[db][4 * g4 + 3] * inv)};
      *(bf16x4*)(ob + off + 32 * db + 8 * g4) = v;
    }
  if (h == 0) {
    float* lse = prefix_rows ? a.lse_p : a.lse_s;
    lse[(size_t)(row_base + my_lp) * a.hq + hq] = (m + log2f(l)) * kLn2;
  }
}

hipError_t launch_fwd_bf16(const AttnArgs& a, int head_dim, int n_z, hipStream_t st) {
  const dim3 grid(a.n_prefix_q_tiles + a.n_suffix_q_tiles, a.hq, n_z);
  if (grid.x == 0 || n_z == 0) return hipSuccess;
  ProfileScope ps("fwd_bf16", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(fwd_bf16_kernel<64>, grid, dim3(kFwdThreads), 0, st, a);
  else
    hipLaunchKernelGGL(fwd_bf16_kernel<128>, grid, dim3(kFwdThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace spr
