// bf16 backward attention on gfx950 matrix cores: Phase B suffix backward
// with gradient-cache accumulation, Phase C prefix backward with cache
// injection, and the dense baseline's backward.
//
// What it computes (paper App. A.2-A.5): with P = exp(S - LSE),
// dP = dO V^T and dS = P * (dP - rowsum(dO * O)) over the joint row,
//   dV = P^T dO,  dK = dS^T Q / sqrt(d),  dQ = dS K / sqrt(d).
// Two kernels split the work so that no gradient needs atomics:
//
// bwd_kv (key-outer): one workgroup owns a 128-key tile of one kv head and
//   sweeps every query row that sees it, for all G q heads of the kv head.
//   For a prefix key tile in Phase B the rows are all suffix rows of the
//   microbatch, so the tile's dK/dV are exactly gK_1 = dS_21^T Q_2 / sqrt(d)
//   and gV_1 = P_21^T dO_2; the workgroup adds them into the fp32 cache
//   G_K/G_V with a plain read-modify-write.  Each (prefix tile, kv head)
//   belongs to exactly one workgroup of a launch, so the cache update is
//   deterministic.  In Phase C the epilogue writes dK_1 = local + G_K and
//   dV_1 = local + G_V instead.  Per 64-row tile and wave (32 keys):
//     S  = Q K^T, dP = dO V^T     A = Q/dO rows (natural tiles), B = K/V (registers)
//     dV += P^T dO, dK += dS^T Q  A = P^T/dS^T from the S/dP registers,
//                                 B = dO/Q columns (transposed tiles)
// bwd_q (query-outer): one workgroup owns 128 query rows of one q head and
//   sweeps their visible key tiles, recomputing S and dP:
//     S^T = K Q^T, dP^T = V dO^T  A = K/V rows (natural tiles), B = Q/dO (registers)
//     dQ^T += K^T dS^T            A = K columns (transposed tile), B = dS^T registers
//   and writes dQ once, already scaled and rounded.
// Both stream their tiles through double-buffered LDS with the next tile's
// global loads in flight during the current tile's products.
#include "common.hpp"
#include "launch.hpp"
#include "tile.hpp"

namespace spr {

namespace {
constexpr int kKvBK = 128;  // keys per bwd_kv workgroup (32 per wave)
constexpr int kKvBQ = 64;   // rows per streamed tile
constexpr int kQBQ = 128;   // rows per bwd_q workgroup (32 per wave)
constexpr int kQBK = 64;    // keys per streamed tile
constexpr int kBwdThreads = 256;
}  // namespace

int bwd_bf16_block_k() { return kKvBK; }

// ---------------------------------------------------------------- bwd_kv
template <int D>
__global__ __launch_bounds__(kBwdThreads) void bwd_kv_bf16_kernel(AttnArgs a) {
  using TG = TileGeom<D>;
  constexpr int BK = kKvBK, BQ = kKvBQ;
  constexpr int NS = D / 16;
  constexpr int NDB = D / 32;
  __shared__ __attribute__((aligned(16))) bf16 Qn[2][TG::NAT];
  __shared__ __attribute__((aligned(16))) bf16 On[2][TG::NAT];  // dO, natural
  __shared__ __attribute__((aligned(16))) bf16 Qt[2][TG::TRN];
  __shared__ __attribute__((aligned(16))) bf16 Ot[2][TG::TRN];  // dO, transposed
  __shared__ __attribute__((aligned(16))) float Ls[2][BQ];
  __shared__ __attribute__((aligned(16))) float Dd[2][BQ];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r = lane & 31, h = lane >> 5;
  const int hk = blockIdx.y, G = a.hq / a.hkv;

  // ---- which 128 keys: a prefix tile, or a tile of suffix s
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
  const int my_key = k0 + 32 * w + r;  // segment-local key of this lane's S/dP column
  const bool kvalid = my_key < kseg;

  // K, V as the B operand of S = Q K^T and dP = dO V^T
  bf16x8 kf[NS], vf[NS];
  {
    const bf16* kg = (const bf16*)(kpre ? a.k_p : a.k_s);
    const bf16* vg = (const bf16*)(kpre ? a.v_p : a.v_s);
    const size_t off = ((size_t)(kbase + (kvalid ? my_key : k0)) * a.hkv + hk) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      kf[s] = kvalid ? *(const bf16x8*)(kg + off + 16 * s) : zero_bf8();
      vf[s] = kvalid ? *(const bf16x8*)(vg + off + 16 * s) : zero_bf8();
    }
  }
  f32x16 dk[NDB], dv[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    dk[db] = zero16();
    dv[db] = zero16();
  }

  // ---- the row tiles this key tile sees, per q head of the group:
  // prefix key tile: prefix rows from k0 on (causal) and/or every suffix row
  // of suffixes seq_base .. seq_base + n_seq - 1 (all visible);
  // suffix key tile: the suffix's own rows from k0 on (causal).
  int n_pr = 0, n_sr = 0, sr0 = 0, sr1 = 0;
  if (kpre) {
    if (a.prefix_rows) n_pr = (a.P - k0 + BQ - 1) / BQ;
    if (a.suffix_rows) {
      sr0 = a.cu[a.seq_base];
      sr1 = a.cu[a.seq_base + a.n_seq];
      n_sr = (sr1 - sr0 + BQ - 1) / BQ;
    }
  } else {
    n_sr = (kseg - k0 + BQ - 1) / BQ;
  }
  const int per_head = n_pr + n_sr;
  const int ntiles = G * per_head;
  struct RowTile {
    int hh, row0, nr, lp_first;
    bool prefix, causal;
  };
  auto tile_info = [&](int t) {
    RowTile rt;
    rt.hh = hk * G + t / per_head;
    const int j = t % per_head;
    if (j < n_pr) {
      rt.prefix = true;
      rt.causal = true;
      rt.lp_first = k0 + j * BQ;
      rt.row0 = rt.lp_first;
      rt.nr = min(BQ, a.P - rt.lp_first);
    } else if (kpre) {
      rt.prefix = false;
      rt.causal = false;
      rt.lp_first = 0;
      rt.row0 = sr0 + (j - n_pr) * BQ;
      rt.nr = min(BQ, sr1 - rt.row0);
    } else {
      rt.prefix = false;
      rt.causal = true;
      rt.lp_first = k0 + j * BQ;
      rt.row0 = kbase + rt.lp_first;
      rt.nr = min(BQ, kseg - rt.lp_first);
    }
    return rt;
  };
  Stager<D> sq, so;
  float lreg = 0.f, dreg = 0.f;
  auto stage_load = [&](int t) {
    const RowTile rt = tile_info(t);
    const bf16* qg = (const bf16*)(rt.prefix ? a.q_p : a.q_s);
    const bf16* dg = (const bf16*)(rt.prefix ? a.do_p : a.do_s);
    sq.load(qg, rt.row0, rt.nr, a.hq, rt.hh, tid);
    so.load(dg, rt.row0, rt.nr, a.hq, rt.hh, tid);
    if (tid < BQ) {
      const float* lg = rt.prefix ? a.lse_p : a.lse_s;
      const float* ddg = rt.prefix ? a.dd_p : a.dd_s;
      const bool v = tid < rt.nr;
      lreg = v ? lg[(size_t)(rt.row0 + tid) * a.hq + rt.hh] * kLog2e : INFINITY;
      dreg = v ? ddg[(size_t)(rt.row0 + tid) * a.hq + rt.hh] : 0.f;
    }
  };
  auto stage_store = [&](int buf) {
    sq.store_nat(Qn[buf], tid);
    sq.store_trn(Qt[buf], tid);
    so.store_nat(On[buf], tid);
    so.store_trn(Ot[buf], tid);
    if (tid < BQ) {
      Ls[buf][tid] = lreg;
      Dd[buf][tid] = dreg;
    }
  };
  if (ntiles > 0) {
    stage_load(0);
    stage_store(0);
  }
  __syncthreads();

  const int q_off = nat_off<D>(r, 0, h);  // A-operand reads: LDS row 32 rb + r
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) stage_load(t + 1);  // global loads in flight during the MFMAs
    const RowTile rt = tile_info(t);
    const bf16* Qb = Qn[buf] + q_off;
    const bf16* Ob = On[buf] + q_off;
    // S = Q K^T and dP = dO V^T for the two 32-row blocks of the tile:
    // acc[rb][i] is tile row 32 rb + c_row(i, h), key my_key
    f32x16 sacc[2], pacc[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      sacc[rb] = zero16();
      pacc[rb] = zero16();
    }
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        sacc[rb] = mfma32(lds8(Qb, nat_off<D>(32 * rb, 16 * s, 0)), kf[s], sacc[rb]);
        pacc[rb] = mfma32(lds8(Ob, nat_off<D>(32 * rb, 16 * s, 0)), vf[s], pacc[rb]);
      }
    // P and dS (softmax backward of the joint row); rows of element i of a
    // block come in runs of 8: 32 rb + 16 (i / 8) + 8 h + i % 8
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int q0 = 32 * rb + 16 * half + 8 * h;
        const float4 l0 = *(const float4*)(&Ls[buf][q0]);
        const float4 l1 = *(const float4*)(&Ls[buf][q0 + 4]);
        const float4 d0 = *(const float4*)(&Dd[buf][q0]);
        const float4 d1 = *(const float4*)(&Dd[buf][q0 + 4]);
        const float lq[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
        const float dq[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const int i = 8 * half + b, q = q0 + b;
          const bool vis = kvalid && q < rt.nr && (!rt.causal || my_key <= rt.lp_first + q);
          const float p = fast_exp2(fmaf(sacc[rb][i], a.scale_log2, -lq[b]));
          const float pv = vis ? p : 0.f;
          sacc[rb][i] = pv;
          pacc[rb][i] = pv * (pacc[rb][i] - dq[b]);
        }
      }
    // dV += P^T dO ; dK += dS^T Q over 16-row steps u: rows 16 u + 8 h + 0..7
#pragma unroll
    for (int u = 0; u < BQ / 16; ++u) {
      const bf16x8 pa = c_to_kfrag(sacc[u >> 1], u & 1);
      const bf16x8 sa = c_to_kfrag(pacc[u >> 1], u & 1);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int off = trn_off(32 * db + r, u, h);
        dv[db] = mfma32(pa, lds8(Ot[buf], off), dv[db]);
        dk[db] = mfma32(sa, lds8(Qt[buf], off), dk[db]);
      }
    }
    compiler_fence();
    if (t + 1 < ntiles) stage_store(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: dk[db][i] is key 32 w + 8 (i/4) + 4 h + i%4, d = 32 db + r
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int key = k0 + 32 * w + 8 * (i >> 2) + 4 * h + (i & 3);
    if (key >= kseg) continue;
    if (kpre) {
      const size_t off = ((size_t)key * a.hkv + hk) * D + r;
      if (a.pk_mode == kPkAccumulate) {
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          a.gk[off + 32 * db] += dk[db][i] * a.scale;
          a.gv[off + 32 * db] += dv[db][i];
        }
      } else {
        bf16* okp = (bf16*)a.dk_p;
        bf16* ovp = (bf16*)a.dv_p;
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          okp[off + 32 * db] = (bf16)(dk[db][i] * a.scale + a.gk[off + 32 * db]);
          ovp[off + 32 * db] = (bf16)(dv[db][i] + a.gv[off + 32 * db]);
        }
      }
    } else {
      const size_t off = ((size_t)(kbase + key) * a.hkv + hk) * D + r;
      bf16* oks = (bf16*)a.dk_s;
      bf16* ovs = (bf16*)a.dv_s;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        oks[off + 32 * db] = (bf16)(dk[db][i] * a.scale);
        ovs[off + 32 * db] = (bf16)dv[db][i];
      }
    }
  }
}

// ----------------------------------------------------------------- bwd_q
template <int D>
__global__ __launch_bounds__(kBwdThreads) void bwd_q_bf16_kernel(AttnArgs a) {
  using TG = TileGeom<D>;
  constexpr int BQ = kQBQ, BK = kQBK;
  constexpr int NS = D / 16;
  constexpr int NDB = D / 32;
  __shared__ __attribute__((aligned(16))) bf16 Kn[2][TG::NAT];
  __shared__ __attribute__((aligned(16))) bf16 Vn[2][TG::NAT];
  __shared__ __attribute__((aligned(16))) bf16 Kt[2][TG::TRN];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r = lane & 31, h = lane >> 5;

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
  const int wave_lp0 = lp0 + 32 * w;
  const int my_lp = wave_lp0 + r;
  const bool row_valid = my_lp < seg_len;

  // Q, dO as the B operands of S^T = K Q^T and dP^T = V dO^T
  bf16x8 qf[NS], df[NS];
  float lse2 = 0.f, drow = 0.f;
  {
    const bf16* qb = (const bf16*)(prefix_rows ? a.q_p : a.q_s);
    const bf16* db = (const bf16*)(prefix_rows ? a.do_p : a.do_s);
    const size_t row = (size_t)(row_base + (row_valid ? my_lp : 0));
    const size_t off = (row * a.hq + hq) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      qf[s] = row_valid ? *(const bf16x8*)(qb + off + 16 * s) : zero_bf8();
      df[s] = row_valid ? *(const bf16x8*)(db + off + 16 * s) : zero_bf8();
    }
    if (row_valid) {
      lse2 = (prefix_rows ? a.lse_p : a.lse_s)[row * a.hq + hq] * kLog2e;
      drow = (prefix_rows ? a.dd_p : a.dd_s)[row * a.hq + hq];
    }
  }
  f32x16 dq[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) dq[db] = zero16();

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
  auto stage_store = [&](int buf) {
    sk.store_nat(Kn[buf], tid);
    sk.store_trn(Kt[buf], tid);
    sv.store_nat(Vn[buf], tid);
  };
  if (ntiles > 0) {
    stage_load(0);
    stage_store(0);
  }
  __syncthreads();

  const int k_off = nat_off<D>(r, 0, h);  // A-operand reads: LDS row 32 kb + r
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) stage_load(t + 1);  // global loads in flight during the MFMAs
    int seg, k0, nk;
    tile_info(t, seg, k0, nk);
    const bool causal = (seg == 0) == prefix_rows;
    if (!(causal && k0 > wave_lp0 + 31)) {  // else no row of this wave sees the tile
      const bf16* Kb = Kn[buf] + k_off;
      const bf16* Vb = Vn[buf] + k_off;
      // st[kb][i] = S^T[key k0 + 32 kb + c_row(i, h)][row my_lp]; pt = dP^T
      f32x16 st[BK / 32], pt[BK / 32];
#pragma unroll
      for (int kb = 0; kb < BK / 32; ++kb) {
        st[kb] = zero16();
        pt[kb] = zero16();
      }
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int kb = 0; kb < BK / 32; ++kb) {
          st[kb] = mfma32(lds8(Kb, nat_off<D>(32 * kb, 16 * s, 0)), qf[s], st[kb]);
          pt[kb] = mfma32(lds8(Vb, nat_off<D>(32 * kb, 16 * s, 0)), df[s], pt[kb]);
        }
      // keys kk < lim are visible to this lane's row
      const int lim = !row_valid ? 0 : (causal ? min(nk, my_lp - k0 + 1) : nk);
#pragma unroll
      for (int kb = 0; kb < BK / 32; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int kk = 32 * kb + c_row(i, h);
          const float p = fast_exp2(fmaf(st[kb][i], a.scale_log2, -lse2));
          pt[kb][i] = kk < lim ? p * (pt[kb][i] - drow) : 0.f;  // dS^T
        }
      // dQ^T += K^T dS^T over 16-key steps u: keys 16 u + 8 h + 0..7
#pragma unroll
      for (int u = 0; u < BK / 16; ++u) {
        const bf16x8 sb = c_to_kfrag(pt[u >> 1], u & 1);
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          dq[db] = mfma32(lds8(Kt[buf], trn_off(32 * db + r, u, h)), sb, dq[db]);
      }
    }
    compiler_fence();
    if (t + 1 < ntiles) stage_store(buf ^ 1);
    __syncthreads();
  }

  if (!row_valid) return;
  // dq[db][i] = dQ^T[d = 32 db + 8 (i/4) + 4 h + i%4][row my_lp] (unscaled)
  const size_t off = ((size_t)(row_base + my_lp) * a.hq + hq) * D + 4 * h;
  if (prefix_rows && a.dq_p_accumulate) {
    // dense baseline: the prefix rows' dQ sums over the trajectories
    float* acc = a.dq_acc_p;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        float4* p4 = (float4*)(acc + off + 32 * db + 8 * g4);
        float4 v = *p4;
        v.x += dq[db][4 * g4];
        v.y += dq[db][4 * g4 + 1];
        v.z += dq[db][4 * g4 + 2];
        v.w += dq[db][4 * g4 + 3];
        *p4 = v;
      }
    return;
  }
  bf16* out = (bf16*)(prefix_rows ? a.dq_p : a.dq_s);
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const bf16x4 v = {(bf16)(dq[db][4 * g4] * a.scale), (bf16)(dq[db][4 * g4 + 1] * a.scale),
                        (bf16)(dq[db][4 * g4 + 2] * a.scale), (bf16)(dq[db][4 * g4 + 3] * a.scale)};
      *(bf16x4*)(out + off + 32 * db + 8 * g4) = v;
    }
}

hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, int n_qz, bool deterministic,
                           hipStream_t st) {
  (void)deterministic;  // both kernels are deterministic: no atomics anywhere
  {
    const dim3 grid(a.n_prefix_k_tiles + a.n_seq * a.n_suffix_k_tiles, a.hkv, 1);
    if (grid.x > 0) {
      ProfileScope ps("bwd_kv_bf16", st);
      if (head_dim == 64)
        hipLaunchKernelGGL(bwd_kv_bf16_kernel<64>, grid, dim3(kBwdThreads), 0, st, a);
      else
        hipLaunchKernelGGL(bwd_kv_bf16_kernel<128>, grid, dim3(kBwdThreads), 0, st, a);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  const dim3 grid(a.n_prefix_q_tiles + a.n_suffix_q_tiles, a.hq, n_qz);
  if (grid.x == 0 || n_qz == 0) return hipSuccess;
  ProfileScope ps("bwd_q_bf16", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(bwd_q_bf16_kernel<64>, grid, dim3(kBwdThreads), 0, st, a);
  else
    hipLaunchKernelGGL(bwd_q_bf16_kernel<128>, grid, dim3(kBwdThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace spr
