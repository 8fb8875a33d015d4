// bf16 backward attention on gfx950 matrix cores: Phase B suffix backward
// with gradient-cache accumulation, Phase C prefix backward with cache
// injection, and the dense baseline's backward.
//
// What it computes (paper App. A.2-A.5), per key tile and kv head, over every
// query row that sees the tile (all G q heads of the kv head):
//   P  = exp(S - LSE),  dP = dO V^T,  dS = P * (dP - rowsum(dO * O))
//   dV += P^T dO,  dK += dS^T Q / sqrt(d),  dQ += dS K / sqrt(d)
// For a prefix key tile in Phase B the rows are every suffix row of the
// microbatch, and the tile's dK/dV are exactly gK_1 = dS_21^T Q_2 / sqrt(d)
// and gV_1 = P_21^T dO_2; the workgroup adds them into the fp32 cache
// G_K/G_V with a plain read-modify-write.  Each (prefix tile, kv head) is
// owned by exactly one workgroup of one launch, so no atomics are needed and
// the cache is bitwise reproducible.  In Phase C the same epilogue writes
// dK_1 = local + G_K and dV_1 = local + G_V instead.
//
// Structure: one workgroup = 4 waves = one 64-key tile; wave w owns keys
// 16 w .. 16 w + 15 and keeps their K/V fragments and dK/dV accumulators in
// registers.  Query rows stream through LDS in tiles of 64 (natural layout).
// Per row tile and wave (16 keys x 64 rows):
//   S  = Q K^T, dP = dO V^T      A = Q/dO rows (LDS), B = K/V (registers)
//   dV += P^T dO, dK += dS^T Q   A = P^T/dS^T straight from the S/dP
//                                registers, B = dO/Q columns via LDS
//                                transpose reads
//   dS^T -> LDS; dQ = dS K       A = dS via transpose reads, B = K columns
//                                (registers); each wave owns d/4 columns and
//                                adds its 64 x d/4 block into an fp32 dQ
//                                accumulator with float atomics.
#include "common.hpp"
#include "launch.hpp"
#include "mfma.hpp"

namespace spr {

namespace {
constexpr int kBwdBK = 64;
constexpr int kBwdBQ = 64;
constexpr int kBwdThreads = 256;
}  // namespace

int bwd_bf16_block_k() { return kBwdBK; }

template <int D>
__global__ __launch_bounds__(kBwdThreads) void bwd_bf16_kernel(AttnArgs a) {
  constexpr int BK = kBwdBK, BQ = kBwdBQ;
  constexpr int NS = D / 32;     // k-steps over d for S and dP
  constexpr int NDB = D / 16;    // d blocks of dK/dV
  constexpr int NQB = BQ / 16;   // row blocks of a row tile
  constexpr int RS = D + 16;     // Q/dO tile row stride (transpose reads conflict-free)
  constexpr int SS = BQ + 16;    // dS^T tile row stride
  constexpr int DQW = D / 4;     // dQ columns owned by one wave
  constexpr int NQN = DQW / 16;
  __shared__ __attribute__((aligned(16))) bf16 Qs[BQ * RS];
  __shared__ __attribute__((aligned(16))) bf16 dOs[BQ * RS];
  __shared__ __attribute__((aligned(16))) bf16 dSt[BK * SS];
  __shared__ float Ls[BQ], Dd[BQ];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c = lane & 15, g = lane >> 4;
  const int hk = blockIdx.y, G = a.hq / a.hkv;

  // ---- which 64 keys: a prefix tile, or a tile of suffix s
  const int x = blockIdx.x;
  bool kpre;
  int k0, kseg, kbase;
  if (x < a.n_prefix_k_tiles) {
    kpre = true;
    k0 = x * BK;
    kseg = a.P;
    kbase = 0;
  } else {
    const int y = x - a.n_prefix_k_tiles;
    const int s = a.seq_base + y / a.n_suffix_k_tiles;
    k0 = (y % a.n_suffix_k_tiles) * BK;
    kbase = a.cu[s];
    kseg = a.cu[s + 1] - kbase;
    kpre = false;
  }
  if (k0 >= kseg) return;
  const bf16* kglob = (const bf16*)(kpre ? a.k_p : a.k_s);
  const bf16* vglob = (const bf16*)(kpre ? a.v_p : a.v_s);
  const int my_key = k0 + 16 * w + c;  // segment-local key of this lane's S/dP column
  const bool kvalid = my_key < kseg;

  // K, V as the B operand of S = Q K^T and dP = dO V^T
  bf16x8 kf[NS], vf[NS];
  {
    const size_t off = ((size_t)(kbase + (kvalid ? my_key : k0)) * a.hkv + hk) * D + 8 * g;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      kf[s] = kvalid ? *(const bf16x8*)(kglob + off + 32 * s) : zero8();
      vf[s] = kvalid ? *(const bf16x8*)(vglob + off + 32 * s) : zero8();
    }
  }
  // K as the B operand of dQ = dS K (slot (g, j) of k-step t holds key
  // 32 t + 4 g + j or 32 t + 16 + 4 g + j - 4; n = this wave's columns):
  // stage the tile in LDS once and read its columns with transpose reads.
  bf16x8 ktf[BK / 32][NQN];
  for (int i = tid; i < BK * (D / 8); i += kBwdThreads) {
    const int r = i / (D / 8), cc = (i % (D / 8)) * 8;
    bf16x8 kv = zero8();
    if (k0 + r < kseg) kv = *(const bf16x8*)(kglob + ((size_t)(kbase + k0 + r) * a.hkv + hk) * D + cc);
    *(bf16x8*)(Qs + r * RS + cc) = kv;
  }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < BK / 32; ++t)
#pragma unroll
    for (int nb = 0; nb < NQN; ++nb)
      ktf[t][nb] = join(lds_col4(Qs, RS, 32 * t + 4 * g, w * DQW + 16 * nb, c),
                        lds_col4(Qs, RS, 32 * t + 16 + 4 * g, w * DQW + 16 * nb, c));

  f32x4 dk[NDB], dv[NDB];
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb) {
    dk[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    dv[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // One tile of up to 64 query rows of head hh: memory rows row0 .. row0+nr-1
  // whose segment-local index is lp_first + r.  `causal`: the rows are in the
  // key tile's own segment, so row r sees key j only if j <= lp_first + r.
  auto row_tile = [&](int hh, bool rows_prefix, int row0, int nr, bool causal, int lp_first) {
    const bf16* qg = (const bf16*)(rows_prefix ? a.q_p : a.q_s);
    const bf16* dg = (const bf16*)(rows_prefix ? a.do_p : a.do_s);
    const float* lg = rows_prefix ? a.lse_p : a.lse_s;
    const float* ddg = rows_prefix ? a.dd_p : a.dd_s;
    float* dqacc = rows_prefix ? a.dq_acc_p : a.dq_acc_s;
    __syncthreads();  // LDS tiles of the previous row tile are consumed
    for (int i = tid; i < BQ * (D / 8); i += kBwdThreads) {
      const int r = i / (D / 8), cc = (i % (D / 8)) * 8;
      bf16x8 qv = zero8(), dv8 = zero8();
      if (r < nr) {
        const size_t off = ((size_t)(row0 + r) * a.hq + hh) * D + cc;
        qv = *(const bf16x8*)(qg + off);
        dv8 = *(const bf16x8*)(dg + off);
      }
      *(bf16x8*)(Qs + r * RS + cc) = qv;
      *(bf16x8*)(dOs + r * RS + cc) = dv8;
    }
    if (tid < BQ) {
      const bool v = tid < nr;
      Ls[tid] = v ? lg[(size_t)(row0 + tid) * a.hq + hh] * kLog2e : INFINITY;
      Dd[tid] = v ? ddg[(size_t)(row0 + tid) * a.hq + hh] : 0.f;
    }
    __syncthreads();

    // S = Q K^T and dP = dO V^T: acc[qb][i] is row 16 qb + 4 g + i, key my_key
    f32x4 sacc[NQB], pacc[NQB];
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      sacc[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
      pacc[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bf16x8 qa = *(const bf16x8*)(Qs + (16 * qb + c) * RS + 32 * s + 8 * g);
        const bf16x8 da = *(const bf16x8*)(dOs + (16 * qb + c) * RS + 32 * s + 8 * g);
        sacc[qb] = mfma16x16x32(qa, kf[s], sacc[qb]);
        pacc[qb] = mfma16x16x32(da, vf[s], pacc[qb]);
      }
    }
    // P and dS (softmax backward of the joint row)
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = 16 * qb + 4 * g + i;
        const bool vis = kvalid && q < nr && (!causal || my_key <= lp_first + q);
        const float p = vis ? exp2f(sacc[qb][i] * a.scale_log2 - Ls[q]) : 0.f;
        sacc[qb][i] = p;
        pacc[qb][i] = p * (pacc[qb][i] - Dd[q]);
      }
    // dV += P^T dO ; dK += dS^T Q  (k = rows, slots as for the keys of dQ)
#pragma unroll
    for (int t = 0; t < NQB / 2; ++t) {
      const bf16x8 pa = pack8(sacc[2 * t], sacc[2 * t + 1]);
      const bf16x8 sa = pack8(pacc[2 * t], pacc[2 * t + 1]);
#pragma unroll
      for (int nb = 0; nb < NDB; ++nb) {
        const bf16x8 dob = join(lds_col4(dOs, RS, 32 * t + 4 * g, 16 * nb, c),
                                lds_col4(dOs, RS, 32 * t + 16 + 4 * g, 16 * nb, c));
        dv[nb] = mfma16x16x32(pa, dob, dv[nb]);
        const bf16x8 qbv = join(lds_col4(Qs, RS, 32 * t + 4 * g, 16 * nb, c),
                                lds_col4(Qs, RS, 32 * t + 16 + 4 * g, 16 * nb, c));
        dk[nb] = mfma16x16x32(sa, qbv, dk[nb]);
      }
    }
    // dS^T[key 16 w + c][rows 16 qb + 4 g .. +3]
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const bf16x4 v = {f2bf(pacc[qb][0]), f2bf(pacc[qb][1]), f2bf(pacc[qb][2]), f2bf(pacc[qb][3])};
      *(bf16x4*)(dSt + (16 * w + c) * SS + 16 * qb + 4 * g) = v;
    }
    __syncthreads();
    // dQ[rows][this wave's columns] += dS K
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      f32x4 acc[NQN];
#pragma unroll
      for (int nb = 0; nb < NQN; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < BK / 32; ++t) {
        const bf16x8 sa = join(lds_col4(dSt, SS, 32 * t + 4 * g, 16 * qb, c),
                               lds_col4(dSt, SS, 32 * t + 16 + 4 * g, 16 * qb, c));
#pragma unroll
        for (int nb = 0; nb < NQN; ++nb) acc[nb] = mfma16x16x32(sa, ktf[t][nb], acc[nb]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = 16 * qb + 4 * g + i;
        if (q < nr) {
          float* dst = dqacc + ((size_t)(row0 + q) * a.hq + hh) * D + w * DQW + c;
#pragma unroll
          for (int nb = 0; nb < NQN; ++nb) unsafeAtomicAdd(dst + 16 * nb, acc[nb][i]);
        }
      }
    }
  };

  for (int hh = hk * G; hh < hk * G + G; ++hh) {
    if (kpre) {
      if (a.prefix_rows)
        for (int rt = k0; rt < a.P; rt += BQ) row_tile(hh, true, rt, min(BQ, a.P - rt), true, rt);
      if (a.suffix_rows) {
        const int r0 = a.cu[a.seq_base], r1 = a.cu[a.seq_base + a.n_seq];
        for (int rt = r0; rt < r1; rt += BQ) row_tile(hh, false, rt, min(BQ, r1 - rt), false, 0);
      }
    } else {
      for (int lr = k0; lr < kseg; lr += BQ)
        row_tile(hh, false, kbase + lr, min(BQ, kseg - lr), true, lr);
    }
  }

  // ---- epilogue: dk[nb][i] / dv[nb][i] belong to key 16 w + 4 g + i, d = 16 nb + c
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int key = k0 + 16 * w + 4 * g + i;
    if (key >= kseg) continue;
    if (kpre) {
      const size_t off = ((size_t)key * a.hkv + hk) * D + c;
      if (a.pk_mode == kPkAccumulate) {
#pragma unroll
        for (int nb = 0; nb < NDB; ++nb) {
          a.gk[off + 16 * nb] += dk[nb][i] * a.scale;
          a.gv[off + 16 * nb] += dv[nb][i];
        }
      } else {
        bf16* okp = (bf16*)a.dk_p;
        bf16* ovp = (bf16*)a.dv_p;
#pragma unroll
        for (int nb = 0; nb < NDB; ++nb) {
          okp[off + 16 * nb] = f2bf(dk[nb][i] * a.scale + a.gk[off + 16 * nb]);
          ovp[off + 16 * nb] = f2bf(dv[nb][i] + a.gv[off + 16 * nb]);
        }
      }
    } else {
      const size_t off = ((size_t)(kbase + key) * a.hkv + hk) * D + c;
      bf16* oks = (bf16*)a.dk_s;
      bf16* ovs = (bf16*)a.dv_s;
#pragma unroll
      for (int nb = 0; nb < NDB; ++nb) {
        oks[off + 16 * nb] = f2bf(dk[nb][i] * a.scale);
        ovs[off + 16 * nb] = f2bf(dv[nb][i]);
      }
    }
  }
}

hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, int n_qz, bool deterministic,
                           hipStream_t st) {
  (void)n_qz;
  if (deterministic) return hipErrorNotSupported;
  const dim3 grid(a.n_prefix_k_tiles + a.n_seq * a.n_suffix_k_tiles, a.hkv, 1);
  if (grid.x == 0) return hipSuccess;
  ProfileScope ps("bwd_bf16", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(bwd_bf16_kernel<64>, grid, dim3(kBwdThreads), 0, st, a);
  else
    hipLaunchKernelGGL(bwd_bf16_kernel<128>, grid, dim3(kBwdThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace spr
