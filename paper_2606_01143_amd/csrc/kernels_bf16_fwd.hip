// bf16 forward attention on gfx950 matrix cores (Phase A prefix forward,
// Phase B suffix forward, and the dense baseline's forward).
//
// What it computes (paper Sec. 3.1 and App. A.1): for each query row,
// O = softmax(S) V over the row's visible keys, S = scale * q k^T, with one
// joint softmax across the prefix keys and the row's own causal suffix keys
// (H_2 = P_21 V_1 + P_22 V_2), plus the row's natural-log LSE.
//
// Structure: one workgroup = 4 waves = 64 query rows of one q head; each
// wave owns 16 rows.  Keys stream in tiles of 64 through LDS in their
// natural row-major layout, first the prefix tiles (read in place from
// K_P/V_P), then the suffix's own tiles; an online softmax carries the row
// max and sum across tiles.  Per tile and wave:
//   S^T (64 keys x 16 rows) = K Q^T   A = K rows from LDS, B = Q in registers
//   O^T (d x 16 rows)      += V^T P^T  A = V columns via LDS transpose reads,
//                                      B = P^T straight from the S^T registers
// Computing S^T rather than S leaves each lane holding 4 keys of one query
// row, which is exactly the B-operand slot layout the PV product needs, so
// P never goes through LDS.
#include "common.hpp"
#include "launch.hpp"
#include "mfma.hpp"

namespace spr {

namespace {
constexpr int kFwdBQ = 64;
constexpr int kFwdBK = 64;
constexpr int kFwdThreads = 256;
}  // namespace

int fwd_bf16_block_q() { return kFwdBQ; }

template <int D>
__global__ __launch_bounds__(kFwdThreads) void fwd_bf16_kernel(AttnArgs a) {
  constexpr int BQ = kFwdBQ, BK = kFwdBK;
  constexpr int NS = D / 32;   // k-steps over d for S^T
  constexpr int NDB = D / 16;  // 16-wide d blocks of O^T
  constexpr int KST = D + 8;   // K tile row stride: 16-byte row reads hit distinct banks
  constexpr int VST = D + 16;  // V tile row stride: transpose reads hit distinct banks
  __shared__ __attribute__((aligned(16))) bf16 Ks[BK * KST];
  __shared__ __attribute__((aligned(16))) bf16 Vs[BK * VST];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c = lane & 15, g = lane >> 4;

  // ---- which 64 query rows: prefix rows, or rows of suffix seq_base + z
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
  const int h = blockIdx.y, hk = h / (a.hq / a.hkv);
  const int wave_lp0 = lp0 + 16 * w;       // first row of this wave
  const int my_lp = wave_lp0 + c;          // this lane's query row (local)
  const bool row_valid = my_lp < seg_len;

  // Q as the B operand of S^T = K Q^T: lane holds Q[my_lp][32 s + 8 g + j]
  bf16x8 qf[NS];
  {
    const bf16* qb = (const bf16*)(prefix_rows ? a.q_p : a.q_s);
    const size_t off = ((size_t)(row_base + (row_valid ? my_lp : 0)) * a.hq + h) * D + 8 * g;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[s] = row_valid ? *(const bf16x8*)(qb + off + 32 * s) : zero8();
  }
  f32x4 o[NDB];
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;  // running max (log2 domain) and sum of row my_lp
  const int last_lp = min(lp0 + BQ, seg_len) - 1;

  for (int seg = 0; seg < 2; ++seg) {
    // seg 0: prefix keys; seg 1: the suffix's own keys (suffix rows only)
    if (seg == 1 && prefix_rows) break;
    const bool causal = (seg == 0) == prefix_rows;  // keys of the row's own segment
    const int nkeys = seg == 0 ? (prefix_rows ? min(a.P, last_lp + 1) : a.P) : last_lp + 1;
    const bf16* kb = (const bf16*)(seg == 0 ? a.k_p : a.k_s);
    const bf16* vb = (const bf16*)(seg == 0 ? a.v_p : a.v_s);
    const int kbase = seg == 0 ? 0 : row_base;
    for (int k0 = 0; k0 < nkeys; k0 += BK) {
      const int nk = min(BK, nkeys - k0);
      __syncthreads();  // previous tile fully consumed
#pragma unroll
      for (int i = tid; i < BK * (D / 8); i += kFwdThreads) {
        const int r = i / (D / 8), cc = (i % (D / 8)) * 8;
        bf16x8 kv = zero8(), vv = zero8();
        if (r < nk) {
          const size_t off = ((size_t)(kbase + k0 + r) * a.hkv + hk) * D + cc;
          kv = *(const bf16x8*)(kb + off);
          vv = *(const bf16x8*)(vb + off);
        }
        *(bf16x8*)(Ks + r * KST + cc) = kv;
        *(bf16x8*)(Vs + r * VST + cc) = vv;
      }
      __syncthreads();
      if (causal && k0 > wave_lp0 + 15) continue;  // no row of this wave sees the tile

      // S^T = K Q^T ; st[kb][i] = S^T[key k0 + 16 kb + 4 g + i][row my_lp]
      f32x4 st[BK / 16];
#pragma unroll
      for (int kb4 = 0; kb4 < BK / 16; ++kb4) {
        st[kb4] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          const bf16x8 ka = *(const bf16x8*)(Ks + (kb4 * 16 + c) * KST + 32 * s + 8 * g);
          st[kb4] = mfma16x16x32(ka, qf[s], st[kb4]);
        }
      }
      // scale into the log2 domain and mask
      const bool need_mask = nk < BK || (causal && k0 + BK - 1 > wave_lp0);
      float mt = -INFINITY;
#pragma unroll
      for (int kb4 = 0; kb4 < BK / 16; ++kb4)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = st[kb4][i] * a.scale_log2;
          if (need_mask) {
            const int kk = kb4 * 16 + 4 * g + i;
            if (kk >= nk || (causal && k0 + kk > my_lp)) v = -INFINITY;
          }
          st[kb4][i] = v;
          mt = fmaxf(mt, v);
        }
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float mn = fmaxf(m, mt);
      const float mu = mn == -INFINITY ? 0.f : mn;
      const float corr = exp2f(m - mu);
      float rs = 0.f;
#pragma unroll
      for (int kb4 = 0; kb4 < BK / 16; ++kb4)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p = exp2f(st[kb4][i] - mu);
          st[kb4][i] = p;
          rs += p;
        }
      rs += __shfl_xor(rs, 16);
      rs += __shfl_xor(rs, 32);
      l = l * corr + rs;
      m = mn;
#pragma unroll
      for (int nb = 0; nb < NDB; ++nb) o[nb] *= corr;

      // O^T += V^T P^T over k-steps of 32 keys: slot (g, j) holds key
      // 32 t + 4 g + j (j < 4) or 32 t + 16 + 4 g + j - 4 (j >= 4)
#pragma unroll
      for (int t = 0; t < BK / 32; ++t) {
        const bf16x8 pb = pack8(st[2 * t], st[2 * t + 1]);
#pragma unroll
        for (int nb = 0; nb < NDB; ++nb) {
          const bf16x8 va = join(lds_col4(Vs, VST, 32 * t + 4 * g, nb * 16, c),
                                 lds_col4(Vs, VST, 32 * t + 16 + 4 * g, nb * 16, c));
          o[nb] = mfma16x16x32(va, pb, o[nb]);
        }
      }
    }
  }

  if (!row_valid) return;
  // o[nb][i] = O^T[d = 16 nb + 4 g + i][row my_lp]
  const float inv = 1.f / l;
  bf16* ob = (bf16*)(prefix_rows ? a.o_p : a.o_s);
  const size_t off = ((size_t)(row_base + my_lp) * a.hq + h) * D + 4 * g;
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb) {
    const bf16x4 v = {f2bf(o[nb][0] * inv), f2bf(o[nb][1] * inv), f2bf(o[nb][2] * inv),
                      f2bf(o[nb][3] * inv)};
    *(bf16x4*)(ob + off + 16 * nb) = v;
  }
  if (g == 0) {
    float* lse = prefix_rows ? a.lse_p : a.lse_s;
    lse[(size_t)(row_base + my_lp) * a.hq + h] = (m + log2f(l)) * kLn2;
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
