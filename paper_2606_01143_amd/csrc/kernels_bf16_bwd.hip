// bf16 backward attention on gfx950 matrix cores: Phase B suffix backward
// with gradient-cache accumulation, Phase C prefix backward with cache
// injection, and the dense baseline's backward.
//
// What it computes (paper App. A.2-A.5): with P = exp(S - LSE),
// dP = dO V^T and dS = P * (dP - rowsum(dO * O)) over the joint row,
//   dV = P^T dO,  dK = dS^T Q / sqrt(d),  dQ = dS K / sqrt(d).
// Two kernels split the work so that no gradient needs atomics:
//
// bwd_kv (key-outer): one workgroup owns a 128-key tile of one kv head (32
//   keys per wave) and sweeps every query row that sees it, for all G q
//   heads of the kv head.  For a prefix key tile in Phase B the rows are all
//   suffix rows of the microbatch, so the tile's dK/dV are exactly
//   gK_1 = dS_21^T Q_2 / sqrt(d) and gV_1 = P_21^T dO_2; the workgroup adds
//   them into the fp32 cache G_K/G_V with a plain read-modify-write.  Each
//   (prefix tile, kv head) belongs to exactly one workgroup of a launch, so
//   the cache update is deterministic.  In Phase C the epilogue writes
//   dK_1 = local + G_K and dV_1 = local + G_V instead.  Per 32-row block and
//   wave (operand conventions in tile.hpp):
//     S  = Q K^T, dP = dO V^T      A = Q/dO tile rows, B = K/V (registers)
//     dV^T += dO^T P, dK^T += Q^T dS  A = dO/Q tiles read transposed,
//                                     B = P/dS straight from the registers
// bwd_q (query-outer): one workgroup owns 128 query rows of one q head and
//   sweeps their visible key tiles, recomputing S and dP:
//     S^T = K Q^T, dP^T = V dO^T   A = K/V tile rows, B = Q/dO (registers)
//     dQ^T += K^T dS^T             A = K tile read transposed, B = dS^T registers
//   and writes dQ once, already scaled and rounded.
// Both stream their tiles through double-buffered LDS, filled by
// direct-to-LDS loads issued one tile ahead of the products.  The loads
// are invisible to the compiler's wait tracking: every tile is read only
// after tile_barrier (vmcnt(0) + workgroup barrier).
#include "common.hpp"
#include "launch.hpp"
#include "tile.hpp"

namespace spr {

namespace {
constexpr int kKvBK = 64;   // keys per key-outer workgroup (two 32-key wave pairs)
constexpr int kQBQ = 128;   // rows per bwd_q workgroup (32 per wave)
}  // namespace

int bwd_bf16_block_k() { return kKvBK; }

// ---------------------------------------------------------------- bwd_kv
// Key-outer role: one workgroup owns 64 keys of one kv head.  Its four waves
// form two pairs, one per 32-key block.  In a pair, the P-wave holds K and
// accumulates dV, the dS-wave holds V and accumulates dK:
//   P-wave:  S = Q K^T, P = exp(S - LSE) (also written to LDS in bf16),
//            dV^T += dO^T P
//   dS-wave: dP = dO V^T, dS = P (dP - rowsum(dO O)) with P read from LDS,
//            dK^T += Q^T dS
// Every product is computed once, and each wave carries half the state of a
// wave that did all four, so two waves fit per SIMD.
template <int D>
__device__ __forceinline__ void bwd_kv_body(const AttnArgs& a, const int bid, bf16 (*Qs)[Tile<D>::ELEMS],
                                            bf16 (*Os)[Tile<D>::ELEMS], float (*Ls)[kTileRows],
                                            float (*Es)[kTileRows], bf16* Px) {
  constexpr int NS = D / 16;
  constexpr int NDB = D / 32;
  constexpr int BQ = kTileRows;
  // Qs/Os: double-buffered tiles of the streamed rows' Q and dO; Ls/Es: their
  // log2-domain LSE and rowsum(dO * O); Px: P of the current tile,
  // [key block][row block][lane][16] bf16

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int r = lane & 31, h = lane >> 5;
  FragOffsets<D> fo;
  fo.init(lane);
  // block b -> kv head b % Hkv (one XCD per kv head), key tile b / Hkv
  const int hk = bid % a.hkv, x = bid / a.hkv;
  const int G = a.hq / a.hkv;

  // ---- which 64 keys: a prefix tile, or a tile of suffix s
  bool kpre;
  int k0, kseg, kbase;
  if (x < a.n_prefix_k_tiles) {
    kpre = true;
    k0 = x * kKvBK;
    kseg = a.P;
    kbase = 0;
  } else {
    const int y = x - a.n_prefix_k_tiles;
    const int s = a.seq_base + y / a.n_suffix_k_tiles;
    k0 = (y % a.n_suffix_k_tiles) * kKvBK;
    kbase = a.cu[s];
    kseg = a.cu[s + 1] - kbase;
    kpre = false;
  }
  if (k0 >= kseg) return;
  const int kb = w >> 1;               // key block of this wave's pair
  const bool pw = (w & 1) == 0;        // P-wave (dV) or dS-wave (dK)
  const int wave_k0 = k0 + 32 * kb;
  const int my_key = min(wave_k0 + r, kseg - 1);  // keys past the end recompute the last one
  bf16* Pblk = Px + kb * (2 * 64 * 16);  // this pair's P exchange, [rb][lane][16]

  // K (P-wave) or V (dS-wave) as the B operand of S = Q K^T / dP = dO V^T
  bf16x8 kvf[NS];
  {
    const bf16* g = (const bf16*)(pw ? (kpre ? a.k_p : a.k_s) : (kpre ? a.v_p : a.v_s));
    const size_t off = ((size_t)(kbase + my_key) * a.hkv + hk) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < NS; ++s) kvf[s] = *(const bf16x8*)(g + off + 16 * s);
  }
  f32x16 acc[NDB];  // dV^T (P-wave) or dK^T (dS-wave), kept in AGPRs
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = zero16();

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
      rt.lp_first = k0 + (j - n_pr) * BQ;
      rt.row0 = kbase + rt.lp_first;
      rt.nr = min(BQ, kseg - rt.lp_first);
    }
    return rt;
  };

  auto issue = [&](int t, bf16* Qd, bf16* Od, float* Ld, float* Ed) {
    const RowTile rt = tile_info(t);
    load_tile<D>(Qd, (const bf16*)(rt.prefix ? a.q_p : a.q_s), rt.row0, rt.nr, a.hq, rt.hh, w, lane);
    load_tile<D>(Od, (const bf16*)(rt.prefix ? a.do_p : a.do_s), rt.row0, rt.nr, a.hq, rt.hh, w, lane);
    if (w == 0) load_row_vec(Ld, (rt.prefix ? a.lse2_p : a.lse2_s) + rt.hh, rt.row0, rt.nr, a.hq, lane);
    if (w == 1) load_row_vec(Ed, (rt.prefix ? a.dd_p : a.dd_s) + rt.hh, rt.row0, rt.nr, a.hq, lane);
  };

  // Row block rb (rows 32 rb + c_row0(i) + 4 h of the tile) against this
  // pair's 32 keys: hidden when a causal tile's rows all precede the keys;
  // masked (rows outside [q_lo, nr) get P = 0) on the diagonal or a ragged end.
  auto hidden = [&](const RowTile& rt, int rb) { return rt.causal && rt.lp_first + 32 * rb + 31 < wave_k0; };
  auto masked = [&](const RowTile& rt, int rb) {
    return rt.nr < 32 * rb + 32 || (rt.causal && rt.lp_first + 32 * rb < wave_k0 + 31);
  };
  // the S or dP product of block rb: A = Q or dO tile rows, B = kvf
  auto product = [&](const bf16* T, int rb) {
    bf16x8 ta[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) ta[k] = row_frag<D>(T, fo, 32 * rb, k);
    f32x16 c = zero16();
#pragma unroll
    for (int k = 0; k < NS; ++k) c = mfma32(ta[k], kvf[k], c);
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int k = 0; k < NS - 4; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    return c;
  };
  // acc += (dO or Q)^T (P or dS) for block rb, operands pb[v] (C-order rows)
  auto accumulate = [&](const bf16* T, int rb, const bf16x8 (&pb)[2]) {
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      bf16x8 at[NDB];
#pragma unroll
      for (int db = 0; db < NDB; ++db) at[db] = tr_frag<D>(T, fo, 32 * rb + 16 * v, db);
#pragma unroll
      for (int db = 0; db < NDB; ++db) mfma32_acc(acc[db], at[db], pb[v]);
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int k = 0; k < NDB - 2; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
  };

  auto compute = [&](int t, const bf16* Qc, const bf16* Oc, const float* Lc, const float* Ec) {
    const RowTile rt = tile_info(t);
    const int q_lo = rt.causal ? my_key - rt.lp_first : 0;  // row lp_first + q sees my_key iff q >= q_lo
    // phase 1: P-wave S -> P (kept as bf16 operands, copied to LDS);
    //          dS-wave dP.  One product call site for both roles.
    bf16x8 pb[2][2];
    f32x16 dpv[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      if (hidden(rt, rb)) continue;
      f32x16 c = product(pw ? Qc : Oc, rb);
      if (pw) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const float4 l4 = *(const float4*)(Lc + 32 * rb + 8 * g4 + 4 * h);
          c[4 * g4 + 0] = fast_exp2(fmaf(c[4 * g4 + 0], a.scale_log2, -l4.x));
          c[4 * g4 + 1] = fast_exp2(fmaf(c[4 * g4 + 1], a.scale_log2, -l4.y));
          c[4 * g4 + 2] = fast_exp2(fmaf(c[4 * g4 + 2], a.scale_log2, -l4.z));
          c[4 * g4 + 3] = fast_exp2(fmaf(c[4 * g4 + 3], a.scale_log2, -l4.w));
        }
        if (masked(rt, rb)) {
          const int lo = q_lo - 32 * rb - 4 * h, hi = rt.nr - 32 * rb - 4 * h;
#pragma unroll
          for (int i = 0; i < 16; ++i) c[i] = (c_row0(i) >= lo && c_row0(i) < hi) ? c[i] : 0.f;
        }
        pb[rb][0] = c_kfrag(c, 0);
        pb[rb][1] = c_kfrag(c, 1);
        bf16x8* px = (bf16x8*)(Pblk + (rb * 64 + lane) * 16);
        px[0] = pb[rb][0];
        px[1] = pb[rb][1];
      } else {
        dpv[rb] = c;
      }
    }
    __syncthreads();  // P of both row blocks visible to the dS-waves
    // phase 2: P-wave dV^T += dO^T P; dS-wave dS -> dK^T += Q^T dS.  One
    // accumulate call site, so the AGPR accumulators are never copied.
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      if (hidden(rt, rb)) continue;
      bf16x8 ops[2];
      if (pw) {
        ops[0] = pb[rb][0];
        ops[1] = pb[rb][1];
      } else {
        const bf16x8* px = (const bf16x8*)(Pblk + (rb * 64 + lane) * 16);
        const bf16x8 p0 = px[0], p1 = px[1];
        f32x16 ds;
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const float4 e4 = *(const float4*)(Ec + 32 * rb + 8 * g4 + 4 * h);
          const float eq[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int i = 4 * g4 + b;
            const float p = (float)(i < 8 ? p0[i] : p1[i - 8]);
            ds[i] = p * (dpv[rb][i] - eq[b]);
          }
        }
        ops[0] = c_kfrag(ds, 0);
        ops[1] = c_kfrag(ds, 1);
      }
      accumulate(pw ? Oc : Qc, rb, ops);
    }
  };

  if (ntiles > 0) issue(0, Qs[0], Os[0], Ls[0], Es[0]);
  tile_barrier();
  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    if (t + 1 < ntiles) issue(t + 1, Qs[cur ^ 1], Os[cur ^ 1], Ls[cur ^ 1], Es[cur ^ 1]);
    compiler_fence();
    compute(t, Qs[cur], Os[cur], Ls[cur], Es[cur]);
    tile_barrier();
  }

  acc_fence();
  // ---- epilogue: acc[db][i] is dV^T or dK^T at d = 32 db + c_row0(i) + 4 h,
  // key wave_k0 + r
  if (wave_k0 + r >= kseg) return;
  const int key = wave_k0 + r;
  const float sc = pw ? 1.f : a.scale;
  if (kpre) {
    const size_t off = ((size_t)key * a.hkv + hk) * D + 4 * h;
    float* cache = pw ? a.gv : a.gk;
    if (a.pk_mode == kPkAccumulate) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          float4* pc = (float4*)(cache + off + 32 * db + 8 * g4);
          float4 c = *pc;
          c.x += acc[db][4 * g4] * sc;
          c.y += acc[db][4 * g4 + 1] * sc;
          c.z += acc[db][4 * g4 + 2] * sc;
          c.w += acc[db][4 * g4 + 3] * sc;
          *pc = c;
        }
    } else {
      bf16* out = (bf16*)(pw ? a.dv_p : a.dk_p);
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const float4 c = *(const float4*)(cache + off + 32 * db + 8 * g4);
          const bf16x4 v = {(bf16)(acc[db][4 * g4] * sc + c.x), (bf16)(acc[db][4 * g4 + 1] * sc + c.y),
                            (bf16)(acc[db][4 * g4 + 2] * sc + c.z), (bf16)(acc[db][4 * g4 + 3] * sc + c.w)};
          *(bf16x4*)(out + off + 32 * db + 8 * g4) = v;
        }
    }
  } else {
    const size_t off = ((size_t)(kbase + key) * a.hkv + hk) * D + 4 * h;
    bf16* out = (bf16*)(pw ? a.dv_s : a.dk_s);
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const bf16x4 v = {(bf16)(acc[db][4 * g4] * sc), (bf16)(acc[db][4 * g4 + 1] * sc),
                          (bf16)(acc[db][4 * g4 + 2] * sc), (bf16)(acc[db][4 * g4 + 3] * sc)};
        *(bf16x4*)(out + off + 32 * db + 8 * g4) = v;
      }
  }
}

// ----------------------------------------------------------------- bwd_q
struct QBlock {
  int tile, z, hq;
};
__device__ __forceinline__ QBlock decode_q_block(const AttnArgs& a, int bid, int ntx) {
  const int G = a.hq / a.hkv;
  int b = bid;
  const int hk = b % a.hkv;
  b /= a.hkv;
  const int gi = b % G;
  b /= G;
  QBlock qb;
  qb.tile = ntx - 1 - b % ntx;  // rows with the most keys first
  qb.z = b / ntx;
  qb.hq = hk * G + gi;
  return qb;
}

template <int D>
__device__ __forceinline__ void bwd_q_body(const AttnArgs& a, const int bid, bf16 (*Ks)[Tile<D>::ELEMS],
                                           bf16 (*Vs)[Tile<D>::ELEMS]) {
  constexpr int NS = D / 16;
  constexpr int NDB = D / 32;
  constexpr int BK = kTileRows;
  // Ks/Vs: double-buffered key tiles

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int r = lane & 31, h = lane >> 5;
  FragOffsets<D> fo;
  fo.init(lane);

  const QBlock blk = decode_q_block(a, bid, a.n_prefix_q_tiles + a.n_suffix_q_tiles);
  const int seq = a.seq_base + blk.z;
  bool prefix_rows;
  int lp0, seg_len, row_base;
  if (blk.tile < a.n_prefix_q_tiles) {
    prefix_rows = true;
    lp0 = blk.tile * kQBQ;
    seg_len = a.P;
    row_base = 0;
  } else {
    prefix_rows = false;
    lp0 = (blk.tile - a.n_prefix_q_tiles) * kQBQ;
    row_base = a.cu[seq];
    seg_len = a.cu[seq + 1] - row_base;
  }
  if (lp0 >= seg_len) return;
  const int hq = blk.hq, hk = hq / (a.hq / a.hkv);
  const int wave_lp0 = lp0 + 32 * w;
  const int row_lp = wave_lp0 + r;
  const bool row_valid = row_lp < seg_len;
  const int my_lp = row_valid ? row_lp : seg_len - 1;

  // Q, dO as the B operands of S^T = K Q^T and dP^T = V dO^T
  bf16x8 qf[NS], df[NS];
  float lse2, drow;
  {
    const bf16* qb = (const bf16*)(prefix_rows ? a.q_p : a.q_s);
    const bf16* dob = (const bf16*)(prefix_rows ? a.do_p : a.do_s);
    const size_t row = (size_t)(row_base + my_lp);
    const size_t off = (row * a.hq + hq) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      qf[s] = *(const bf16x8*)(qb + off + 16 * s);
      df[s] = *(const bf16x8*)(dob + off + 16 * s);
    }
    lse2 = (prefix_rows ? a.lse2_p : a.lse2_s)[row * a.hq + hq];
    drow = (prefix_rows ? a.dd_p : a.dd_s)[row * a.hq + hq];
  }
  f32x16 dq[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) dq[db] = zero16();

  const int last_lp = min(lp0 + kQBQ, seg_len) - 1;
  const int nkeys0 = prefix_rows ? min(a.P, last_lp + 1) : a.P;
  const int nkeys1 = prefix_rows ? 0 : last_lp + 1;
  const int nt0 = (nkeys0 + BK - 1) / BK, nt1 = (nkeys1 + BK - 1) / BK;
  const int ntiles = nt0 + nt1;

  auto issue = [&](int t, bf16* Kd, bf16* Vd) {
    const int seg = t < nt0 ? 0 : 1;
    const int k0 = (seg == 0 ? t : t - nt0) * BK;
    const int nk = min(BK, (seg == 0 ? nkeys0 : nkeys1) - k0);
    const int kbase = seg == 0 ? 0 : row_base;
    load_tile<D>(Kd, (const bf16*)(seg == 0 ? a.k_p : a.k_s), kbase + k0, nk, a.hkv, hk, w, lane);
    load_tile<D>(Vd, (const bf16*)(seg == 0 ? a.v_p : a.v_s), kbase + k0, nk, a.hkv, hk, w, lane);
  };

  auto compute = [&](int t, const bf16* Kc, const bf16* Vc) {
    const int seg = t < nt0 ? 0 : 1;
    const int k0 = (seg == 0 ? t : t - nt0) * BK;
    const int nk = min(BK, (seg == 0 ? nkeys0 : nkeys1) - k0);
    const bool causal = (seg == 0) == prefix_rows;
    if (causal && k0 > wave_lp0 + 31) return;  // no row of this wave sees the tile
    // st[kb][i] = S^T[key k0 + 32 kb + c_row0(i) + 4 h][row my_lp]; pt = dP^T
    f32x16 st[2] = {zero16(), zero16()}, pt[2] = {zero16(), zero16()};
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        st[kb] = mfma32(row_frag<D>(Kc, fo, 32 * kb, s), qf[s], st[kb]);
        pt[kb] = mfma32(row_frag<D>(Vc, fo, 32 * kb, s), df[s], pt[kb]);
      }
    const bool need_mask = nk < BK || (causal && k0 + BK - 1 > wave_lp0);
    const int lim = (causal ? min(nk, my_lp - k0 + 1) : nk) - 4 * h;  // keys c_row0 + 4 h < lim + 4 h are visible
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) st[kb][i] = fast_exp2(fmaf(st[kb][i], a.scale_log2, -lse2));
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) st[kb][i] = 32 * kb + c_row0(i) < lim ? st[kb][i] : 0.f;
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) pt[kb][i] = st[kb][i] * (pt[kb][i] - drow);  // dS^T
    // dQ^T += K^T dS^T over 16-key steps u (C-order keys)
#pragma unroll
    for (int u = 0; u < BK / 16; ++u) {
      const bf16x8 sb = c_kfrag(pt[u >> 1], u & 1);
#pragma unroll
      for (int db = 0; db < NDB; ++db) dq[db] = mfma32(tr_frag<D>(Kc, fo, 16 * u, db), sb, dq[db]);
    }
  };

  if (ntiles > 0) issue(0, Ks[0], Vs[0]);
  tile_barrier();
  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    if (t + 1 < ntiles) issue(t + 1, Ks[cur ^ 1], Vs[cur ^ 1]);
    compiler_fence();
    compute(t, Ks[cur], Vs[cur]);
    tile_barrier();
  }

  if (!row_valid) return;
  // dq[db][i] = dQ^T[d = 32 db + c_row0(i) + 4 h][row my_lp] (unscaled)
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

// One launch runs both kernels' workgroups: the first n_first blocks take
// one role, the rest the other, so that the key-outer and query-outer work
// of a microbatch share the GPU (a suffix microbatch alone fills neither).
// The heavier role goes first; both segments start on a multiple of 8 blocks
// so the XCD mapping of each role holds.
template <int D>
__global__ __launch_bounds__(kThreads, 2) void bwd_bf16_kernel(AttnArgs a, int n_first, int n_kv,
                                                               int n_q, int kv_first) {
  constexpr int TE = Tile<D>::ELEMS;
  __shared__ __attribute__((aligned(1024))) bf16 tiles[4][TE];
  __shared__ __attribute__((aligned(256))) float rowv[4][kTileRows];
  __shared__ __attribute__((aligned(1024))) bf16 pex[2 * 2 * 64 * 16];
  const int b = blockIdx.x;
  const bool first = b < n_first;
  const int bid = first ? b : b - n_first;
  // the first segment is padded to a multiple of 8 blocks: padding exits
  if (first == (kv_first != 0)) {
    if (bid < n_kv) bwd_kv_body<D>(a, bid, tiles, tiles + 2, rowv, rowv + 2, pex);
  } else {
    if (bid < n_q) bwd_q_body<D>(a, bid, tiles, tiles + 2);
  }
}

hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, int n_qz, bool deterministic,
                           hipStream_t st) {
  (void)deterministic;  // both roles are deterministic: no atomics anywhere
  const long n_kv = (long)(a.n_prefix_k_tiles + a.n_seq * a.n_suffix_k_tiles) * a.hkv;
  const long n_q = (long)(a.n_prefix_q_tiles + a.n_suffix_q_tiles) * a.hq * n_qz;
  if (n_kv + n_q == 0) return hipSuccess;
  // Phase C / dense prefix: the causal key tiles near the start of the prefix
  // carry the most rows; Phase B suffix: every query tile sweeps the prefix
  const int kv_first = a.prefix_rows ? 1 : 0;
  const long first = kv_first ? n_kv : n_q;
  const long n_first = (first + 7) / 8 * 8;
  const long nb = n_first + (kv_first ? n_q : n_kv);
  ProfileScope ps("bwd_bf16", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(bwd_bf16_kernel<64>, dim3((unsigned)nb), dim3(kThreads), 0, st, a, (int)n_first,
                       (int)n_kv, (int)n_q, kv_first);
  else
    hipLaunchKernelGGL(bwd_bf16_kernel<128>, dim3((unsigned)nb), dim3(kThreads), 0, st, a, (int)n_first,
                       (int)n_kv, (int)n_q, kv_first);
  return hipGetLastError();
}

}  // namespace spr
