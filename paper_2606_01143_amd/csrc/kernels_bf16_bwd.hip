// bf16 backward attention on gfx950 matrix cores: Phase B suffix backward
// with gradient-cache accumulation, Phase C prefix backward with cache
// injection, and the dense baseline's backward.
//
// What it computes (paper App. A.2-A.5): with P = exp(S - LSE),
// dP = dO V^T and dS = P * (dP - rowsum(dO * O)) over the joint row,
//   dV = P^T dO,  dK = dS^T Q / sqrt(d),  dQ = dS K / sqrt(d).
// Two workgroup roles split the work so that, by default, no gradient needs
// atomics (with SPR_ATOMIC_DQ the key-outer role also adds dQ, see below):
//
// bwd_kv (key-outer): one workgroup owns a 64-key tile of one kv head, as
//   two wave pairs of 32 keys, and sweeps every query row that sees it, for
//   all G q heads of the kv head.  For a prefix key tile in Phase B the rows are all
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
// Both stream their tiles through LDS (the key-outer role's 32-row Q/dO
// tiles triple-buffered, four buffers in its key-outer-only launch; the
// query-outer role's 64-key K/V tiles double-buffered), filled by
// direct-to-LDS loads issued one tile ahead of the products.  The loads are invisible to the compiler's wait tracking:
// every tile is read only after tile_barrier (vmcnt(0) + workgroup barrier).
#include <algorithm>
#include <cmath>

#include "common.hpp"
#include "launch.hpp"
#include "tile.hpp"

namespace spr {

namespace {
constexpr int kKvBK = 64;   // keys per key-outer workgroup (two 32-key wave pairs)
constexpr int kKvWidePairs = 6;  // wave pairs of the key-outer-only workgroup
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
//
// The rows stream through LDS in 32-row tiles.  The dS-wave runs one tile
// behind its P-wave: between two workgroup barriers the P-wave takes tile t
// (product, exp, P to LDS, accumulate) while the dS-wave takes tile t - 1
// (product, P from LDS, dS, accumulate).  Both waves then do the same kind
// and amount of work per barrier interval, and one barrier per tile both
// publishes P and retires a buffer.  Tiles t - 1 and t are read while tile
// t + 1 loads, so the Q/dO tiles are triple-buffered, and P is
// double-buffered.
namespace {
constexpr int kKvBQ = 32;  // rows per key-outer tile
constexpr int kKvBufs = 3;
}  // namespace

typedef __attribute__((address_space(1))) float gfloat;  // global memory
template <bool B>
struct StepOrder {
  static constexpr bool value = B;
};

// In the key-outer-only launch a deferring dS-wave (below) still reads tile
// t - 2 while tile t + 1 loads: a fourth buffer.
template <int D, bool AQ, int NP = 2>
struct KvLds {
  static constexpr int TE = kKvBQ * D;  // bf16 elements of one 32-row tile
  static constexpr int NB = NP > 2 ? 4 : kKvBufs;
  bf16 q[NB][TE];
  bf16 o[NB][TE];
  float l[NB][64];  // log2-domain LSE of the tile's rows (32 used)
  float e[NB][64];  // rowsum(dO * O) of the tile's rows (32 used)
  bf16x8 p[2][NP][2][64];  // P exchange (bf16) [tile parity][key block][k-step v][lane]
};
template <int D>
struct KvLds<D, true, 2> : KvLds<D, false, 2> {
  // dS^T of a tile for the dQ product: 64 keys x 32 rows bf16, [tile parity]
  bf16 ds[2][64 * kKvBQ];
};

// dS^T exchange tile (64 keys x 32 rows, row-major by key): 16-byte chunk c
// of key row k sits at chunk c ^ ((k >> 2) & 3).  A dS-wave's 8-byte writes
// (32 keys at one column) then spread over all banks, and the transposed
// reads (4 consecutive keys x 32 bytes per 16 lanes) stay conflict-free.
__device__ __forceinline__ int dst_off(int key, int col) {
  return key * kKvBQ + ((((col >> 3) ^ ((key >> 2) & 3))) << 3) + (col & 7);
}

// NP wave pairs (32 keys each) per workgroup: 2 in the launch shared with
// the query-outer role, kKvWidePairs in the key-outer-only launch of long
// prefixes.  PC: the launch is a Phase C (prefix key tiles, causal prefix
// rows only), known at compile time, so the per-tile bookkeeping drops the
// suffix-row cases; in the key-outer-only launch the twelve waves' scalar
// instructions compete for the CU's scalar unit.
template <int D, bool AQ, int NP = 2, bool PC = false>
__device__ __forceinline__ void bwd_kv_body(const AttnArgs& a, const int bid, KvLds<D, AQ, NP>& L) {
  static_assert(NP == 2 || !AQ, "the atomic-dQ variant runs two pairs");
  static_assert(!PC || (NP > 2 && !AQ), "the Phase C form is the key-outer-only launch's");
  constexpr int NB = KvLds<D, AQ, NP>::NB;
  constexpr int NS = D / 16;
  constexpr int NDB = D / 32;
  constexpr int BQ = kKvBQ;
  constexpr int KB = 32 * NP;  // keys per workgroup

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int r = lane & 31, h = lane >> 5;
  FragOffsets<D> fo;
  fo.init(lane);
  // block b -> kv head b % Hkv (one XCD per kv head), row share, key tile
  const int R = a.kv_rsplit > 1 ? a.kv_rsplit : 1;
  const int hk = bid % a.hkv, rs = (bid / a.hkv) % R, x = bid / a.hkv / R;
  const int G = a.hq / a.hkv;

  // ---- which KB keys: a prefix tile, or a tile of suffix s.  Launches
  // without prefix rows take the suffix key tiles first: the causal tiles at
  // the start of a suffix carry about as many rows as a prefix tile, and the
  // shorter ones should not start last.
  const int n_sfx = PC ? 0 : a.n_seq * a.n_suffix_k_tiles;
  const bool sfx_first = !PC && !a.prefix_rows;
  bool kpre;
  int k0, kseg, kbase;
  if (PC || (sfx_first ? x >= n_sfx : x < a.n_prefix_k_tiles)) {
    kpre = true;
    k0 = (sfx_first ? x - n_sfx : x) * KB;
    kseg = a.P;
    kbase = 0;
  } else {
    const int y = sfx_first ? x : x - a.n_prefix_k_tiles;
    const int s = a.seq_base + y / a.n_suffix_k_tiles;
    k0 = (y % a.n_suffix_k_tiles) * KB;
    const SegRows sg = suffix_rows(a.cu, s, a.total_len);
    kbase = sg.base;
    kseg = sg.len;
    kpre = false;
  }
  if (k0 >= kseg) return;
  const int kb = w >> 1;               // key block of this wave's pair
  // P-wave (dV) or dS-wave (dK).  A workgroup's waves take the CU's four
  // SIMDs in a fixed cycle from some starting SIMD, so waves w, w + 4 and
  // w + 8 share one.  Only the P-waves evaluate exp2: in the twelve-wave
  // launch pairs 4 and 5 swap roles, and every SIMD holds both kinds.
  const bool pw = ((w & 1) == 0) != (NP > 2 && w >= 8);
  // Every wave leaves the tile barrier at the same time, so waves taking the
  // same steps in the same order all want the matrix cores at once, then
  // all the vector ALU.  In the key-outer-only launch each SIMD holds two
  // waves of one role and one of the other; that one (waves 8-11) defers
  // each tile's accumulation to the next barrier interval and runs it first
  // there, so its matrix work overlaps the other two waves' elementwise
  // steps.
  const bool defer = NP > 2 && (w >> 2) == 2;
  const int wave_k0 = k0 + 32 * kb;
  const int my_key = min(wave_k0 + r, kseg - 1);  // keys past the end recompute the last one

  // K (P-wave) or V (dS-wave) as the B operand of S = Q K^T / dP = dO V^T
  bf16x8 kvf[NS];
  {
    const bf16* g = (const bf16*)(pw ? (kpre ? a.k_p : a.k_s) : (kpre ? a.v_p : a.v_s));
    const size_t off = ((size_t)(kbase + my_key) * a.hkv + hk) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < NS; ++s) kvf[s] = *(const bf16x8*)(g + off + 16 * s);
#pragma unroll
    for (int s = 0; s < NS; ++s) settle(kvf[s]);
  }
  f32x16 acc[NDB];  // dV^T (P-wave) or dK^T (dS-wave)
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = zero16();
  // the block's last key tile of its segment may be partial: keys past the
  // end recompute the last key and their P must be zero wherever dQ sums
  // over keys
  const bool kpartial = k0 + KB > kseg;
  const bool key_ok = wave_k0 + r < kseg;
  // atomic dQ: wave w < NDB owns dQ columns 32 w .. 32 w + 31 of every row
  // tile; its B operands K[16 v + k][32 w + r] for the 4 k-steps over the
  // block's 64 keys stay in registers for the whole sweep
  const bool dq_on = AQ && a.dq_atomic;
  bf16x8 kq[4];

  // ---- the 32-row tiles this key tile sees, per q head of the group:
  // prefix key tile: prefix rows from k0 on (causal) and/or every suffix row
  // of suffixes seq_base .. seq_base + n_seq - 1 (all visible);
  // suffix key tile: the suffix's own rows from k0 on (causal).
  int n_pr = 0, n_sr = 0, sr0 = 0, sr1 = 0;
  if (PC) {
    n_pr = (a.P - k0 + BQ - 1) / BQ;
  } else if (kpre) {
    if (a.prefix_rows) n_pr = (a.P - k0 + BQ - 1) / BQ;
    if (a.suffix_rows) {
      const SegRows sp = suffix_span(a.cu, a.seq_base, a.seq_base + a.n_seq, a.total_len);
      sr0 = sp.base;
      sr1 = sp.base + sp.len;
      n_sr = (sr1 - sr0 + BQ - 1) / BQ;
    }
  } else {
    n_sr = (kseg - k0 + BQ - 1) / BQ;
  }
  const int per_head = n_pr + n_sr;
  // this block's contiguous share of the (row tile, head) sequence below
  const int t_lo = (int)((long)G * per_head * rs / R);
  const int ntiles = (int)((long)G * per_head * (rs + 1) / R) - t_lo;
  struct RowTile {
    int hh, row0, nr, lp_first;
    bool prefix, causal;
  };
  // Tile order: row tiles outer, the G q heads inner.  The suffix rows of a
  // prefix key tile (all visible) go first, in ascending order; causal row
  // ranges go from the last row tile down to the diagonal.  The key tiles of
  // one kv head run concurrently on one XCD and share the same 32-row grid,
  // so in this order they read each Q/dO row tile at about the same time and
  // it is fetched from HBM once for all of them (swept from each tile's own
  // diagonal upward they drift apart and thrash the L2).
  // The loop keeps (row tile, head) cursors instead of dividing a flat
  // index: every wave of the CU leaves a barrier at once, and their
  // divisions would queue on the shared scalar unit.
  struct Cursor {
    int j, g, buf;  // row tile, q head of the group, LDS buffer
  };
  auto advance = [&](Cursor& c) {
    if (++c.g == G) {
      c.g = 0;
      ++c.j;
    }
    c.buf = c.buf == NB - 1 ? 0 : c.buf + 1;
  };
  auto tile_info = [&](const Cursor& c) {
    RowTile rt;
    rt.hh = hk * G + c.g;
    const int j = c.j;
    if constexpr (PC) {
      rt.prefix = true;
      rt.causal = true;
      rt.lp_first = k0 + (n_pr - 1 - j) * BQ;
      rt.row0 = rt.lp_first;
      rt.nr = min(BQ, a.P - rt.lp_first);
      return rt;
    }
    if (kpre && j < n_sr) {
      rt.prefix = false;
      rt.causal = false;
      rt.lp_first = 0;
      rt.row0 = sr0 + j * BQ;
      rt.nr = min(BQ, sr1 - rt.row0);
    } else if (kpre) {
      rt.prefix = true;
      rt.causal = true;
      rt.lp_first = k0 + (n_pr - 1 - (j - n_sr)) * BQ;
      rt.row0 = rt.lp_first;
      rt.nr = min(BQ, a.P - rt.lp_first);
    } else {
      rt.prefix = false;
      rt.causal = true;
      rt.lp_first = k0 + (n_sr - 1 - j) * BQ;
      rt.row0 = kbase + rt.lp_first;
      rt.nr = min(BQ, kseg - rt.lp_first);
    }
    return rt;
  };

  // tile t's loads, split over waves 0-3
  const bf16 *q_p = in_sgpr((const bf16*)a.q_p), *q_s = in_sgpr((const bf16*)a.q_s);
  const bf16 *do_p = in_sgpr((const bf16*)a.do_p), *do_s = in_sgpr((const bf16*)a.do_s);
  const float *l_p = in_sgpr((const float*)a.lse2_p), *l_s = in_sgpr((const float*)a.lse2_s);
  const float *e_p = in_sgpr((const float*)a.dd_p), *e_s = in_sgpr((const float*)a.dd_s);
  TileLoader<D, 4, BQ> tl;
  tl.init(a.hq, w & 3, lane);
  RowVecLoader rl;
  rl.init(a.hq, lane);
  auto issue = [&](const Cursor& cur) {
    if (NP > 2 && w >= 4) return;  // waves 0-3 load every tile
    const RowTile rt = tile_info(cur);
    const int b = cur.buf;
    tl.load(L.q[b], PC ? q_p : pick(rt.prefix, q_p, q_s), rt.row0, rt.nr, a.hq, rt.hh);
    tl.load(L.o[b], PC ? do_p : pick(rt.prefix, do_p, do_s), rt.row0, rt.nr, a.hq, rt.hh);
    if (w == 0) rl.load(L.l[b], (PC ? l_p : pick(rt.prefix, l_p, l_s)) + rt.hh, rt.row0, rt.nr, a.hq);
    if (w == 1) rl.load(L.e[b], (PC ? e_p : pick(rt.prefix, e_p, e_s)) + rt.hh, rt.row0, rt.nr, a.hq);
  };

  // A tile whose rows all precede this pair's keys (causal) contributes
  // nothing: both waves of the pair skip it.  Masked (rows outside
  // [q_lo, nr) get P = 0): the diagonal tile or a ragged end.
  auto hidden = [&](const RowTile& rt) { return rt.causal && rt.lp_first + BQ - 1 < wave_k0; };
  auto masked = [&](const RowTile& rt) {
    return rt.nr < BQ || (rt.causal && rt.lp_first < wave_k0 + 31) || kpartial;
  };
  // S or dP of the tile: A = Q or dO tile rows, B = kvf
  auto product = [&](const bf16* T) {
    bf16x8 ta[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) ta[k] = row_frag<D>(T, fo, 0, k);
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
  // acc += (dO or Q)^T (P or dS), operands pb[v] (C-order rows).  In the
  // key-outer-only launch a wave raises its issue priority for these eight
  // products, so the SIMD's arbiter feeds the matrix core from it first.
  auto accumulate = [&](const bf16* T, const bf16x8 (&pb)[2]) {
    if constexpr (NP > 2) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      bf16x8 at[NDB];
#pragma unroll
      for (int db = 0; db < NDB; ++db) at[db] = tr_frag<D>(T, fo, 16 * v, db);
#pragma unroll
      for (int db = 0; db < NDB; ++db) acc[db] = mfma32(at[db], pb[v], acc[db]);
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int k = 0; k < NDB - 2; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
    if constexpr (NP > 2) __builtin_amdgcn_s_setprio(0);
  };

  // this wave's work on tile tc: one product and the role's elementwise
  // step (front), giving the bf16 operands of one accumulation (back)
  struct Ops {
    bf16x8 v[2];
  };
  auto front = [&](int tc, const RowTile& rt, const int b) {
    const bf16* Qc = L.q[b];
    const bf16* Oc = L.o[b];
    bf16x8* px = &L.p[tc & 1][kb][0][lane];  // k-step v at px[64 v]
    f32x16 c = product(pw ? Qc : Oc);
    Ops res;
    bf16x8(&ops)[2] = res.v;
    if (pw) {
      const float* Lc = L.l[b];
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const float4 l4 = *(const float4*)(Lc + 8 * g4 + 4 * h);
        c[4 * g4 + 0] = fast_exp2(fmaf(c[4 * g4 + 0], a.scale_log2, -l4.x));
        c[4 * g4 + 1] = fast_exp2(fmaf(c[4 * g4 + 1], a.scale_log2, -l4.y));
        c[4 * g4 + 2] = fast_exp2(fmaf(c[4 * g4 + 2], a.scale_log2, -l4.z));
        c[4 * g4 + 3] = fast_exp2(fmaf(c[4 * g4 + 3], a.scale_log2, -l4.w));
      }
      if (masked(rt)) {
        // row lp_first + q sees my_key iff q >= q_lo; keys past the segment
        // see no row
        const int q_lo = rt.causal ? my_key - rt.lp_first : 0;
        const int lo = q_lo - 4 * h, hi = key_ok ? rt.nr - 4 * h : -1;
#pragma unroll
        for (int i = 0; i < 16; ++i) c[i] = (c_row0(i) >= lo && c_row0(i) < hi) ? c[i] : 0.f;
      }
      ops[0] = c_kfrag(c, 0);
      ops[1] = c_kfrag(c, 1);
      // the bf16 operands of dV^T += dO^T P also go to the dS-wave
      px[0] = ops[0];
      px[64] = ops[1];
    } else {
      // P of this tile was written by the P-wave one barrier ago
      const float* Ec = L.e[b];
      f32x16 ds;
      const bf16x8 pv[2] = {px[0], px[64]};  // C elements 8 v .. 8 v + 7
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const float4 e4 = *(const float4*)(Ec + 8 * g4 + 4 * h);
        const int v = g4 >> 1, j0 = 4 * (g4 & 1);
        ds[4 * g4 + 0] = (float)pv[v][j0 + 0] * (c[4 * g4 + 0] - e4.x);
        ds[4 * g4 + 1] = (float)pv[v][j0 + 1] * (c[4 * g4 + 1] - e4.y);
        ds[4 * g4 + 2] = (float)pv[v][j0 + 2] * (c[4 * g4 + 2] - e4.z);
        ds[4 * g4 + 3] = (float)pv[v][j0 + 3] * (c[4 * g4 + 3] - e4.w);
      }
      ops[0] = c_kfrag(ds, 0);
      ops[1] = c_kfrag(ds, 1);
      if constexpr (AQ) {
        if (dq_on) {
          // dS^T rows 32 kb + r (keys), columns 8 g + 4 h .. + 3 (rows)
          bf16* dsx = L.ds[tc & 1];
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const bf16x8& o8 = ops[g4 >> 1];
            const int j0 = 4 * (g4 & 1);
            *(bf16x4*)(dsx + dst_off(32 * kb + r, 8 * g4 + 4 * h)) =
                bf16x4{o8[j0], o8[j0 + 1], o8[j0 + 2], o8[j0 + 3]};
          }
        }
      }
    }
    return res;
  };
  auto back = [&](const int b, const Ops& o) { accumulate(pw ? L.o[b] : L.q[b], o.v); };

  // dQ of tile tq (atomic variant): dQ[row][32 w + r] += sum over the
  // block's 64 keys of dS[row][key] K[key][32 w + r], A = dS^T read
  // transposed from the exchange tile, B = kq; then one fp32 atomic add per
  // element into the row's accumulator (unscaled; the caller converts).
  // Key blocks whose pair skipped the tile (rows all above its keys) are
  // skipped here too: their exchange tile was not written.
  int trlo = 0, trhi = 0;
  if (dq_on) {
    const int i16 = lane & 15;
    const int col = (lane & 16) + 4 * (i16 & 3);
    trlo = dst_off(4 * h + (i16 >> 2), col);
    trhi = dst_off(8 + 4 * h + (i16 >> 2), col);
  }
  float *dqa_p = nullptr, *dqa_s = nullptr;
  if (dq_on) {
    dqa_p = in_sgpr(a.dq_acc_p);
    dqa_s = in_sgpr(a.dq_acc_s);
  }
  auto dq_step = [&](int tq, const RowTile& rt) {
    if constexpr (AQ) {
      const bool skip0 = rt.causal && rt.lp_first + BQ - 1 < k0;
      const bool skip1 = rt.causal && rt.lp_first + BQ - 1 < k0 + 32;
      if (skip0 || w >= NDB) return;
      const bf16* dsx = L.ds[tq & 1];
      auto ds_frag = [&](int v) {
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(dsx + 16 * v * kKvBQ + trlo));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(dsx + 16 * v * kKvBQ + trhi));
        return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      };
      f32x16 c = zero16();
      c = mfma32(ds_frag(0), kq[0], c);
      c = mfma32(ds_frag(1), kq[1], c);
      if (!skip1) {
        c = mfma32(ds_frag(2), kq[2], c);
        c = mfma32(ds_frag(3), kq[3], c);
      }
      gfloat* base = (gfloat*)pick(rt.prefix, dqa_p, dqa_s) + ((size_t)rt.row0 * a.hq + rt.hh) * D + 32 * w + r;
      const size_t rs = (size_t)a.hq * D;  // row stride
      if (rt.nr >= BQ) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
          __builtin_amdgcn_global_atomic_fadd_f32(base + (size_t)(c_row0(i) + 4 * h) * rs, c[i]);
      } else {
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (c_row0(i) + 4 * h < rt.nr)
            __builtin_amdgcn_global_atomic_fadd_f32(base + (size_t)(c_row0(i) + 4 * h) * rs, c[i]);
      }
    }
  };


  // iteration t: the P-wave takes tile t, the dS-wave tile t - 1; tile t + 1
  // loads meanwhile
  Cursor cl = {t_lo / G, t_lo % G, 0};  // next tile to load
  Cursor cc = cl;                        // next tile this wave computes
  Cursor cq = cl;                        // next tile whose dQ this wave adds
  if (ntiles > 0) {
    issue(cl);
    advance(cl);
  }
  if (dq_on) {
    // the block's 64 keys, staged once through Q/dO buffers 1-2 (free until
    // the first iteration loads tile 1), then read as the dQ product's B
    // operands; keys past the segment repeat the last one
    const bf16* kb_ = (const bf16*)(kpre ? a.k_p : a.k_s);
    load_tile<D, 4, kKvBK>(&L.q[1][0], kb_, kbase + k0, kseg - k0, a.hkv, hk, w, lane);
  }
  tile_barrier();
  if (dq_on) {
    if (w < NDB) {
      // K[16 v + k][32 w + r]: the transposed read of tr_frag at column
      // block w (a wave-uniform index, so the offsets are formed here)
      const int i16 = lane & 15, col = 32 * w + (lane & 16) + 4 * (i16 & 3);
      const int olo = toff<D>(4 * h + (i16 >> 2), col), ohi = toff<D>(8 + 4 * h + (i16 >> 2), col);
      const bf16* kt = &L.q[1][0];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(kt + 16 * v * D + olo));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(kt + 16 * v * D + ohi));
        kq[v] = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) settle(kq[v]);
    }
    __syncthreads();  // every wave holds its operands before buffer 1 reloads
  }
  const int t_end = dq_on ? ntiles + 1 : ntiles;
  // The tile loop, in one of two step orders fixed at compile time (the
  // deferring order carries one tile's operands across the barrier; compiled
  // as one loop with a runtime order, those registers would stay live through
  // every wave's products).
  auto sweep = [&](auto order) {
    constexpr bool DEFER = decltype(order)::value;
    // a deferring wave's accumulation still to do: tile buffer and operands
    bool pend = false;
    int pend_buf = 0;
    Ops pend_ops;
    for (int t = 0; t <= t_end; ++t) {
      if (t + 1 < ntiles) {
        issue(cl);
        advance(cl);
      }
      compiler_fence();
      const int tc = pw ? t : t - 1;
      if constexpr (DEFER) {
        if (pend) back(pend_buf, pend_ops);
        pend = false;
      }
      if (tc >= 0 && tc < ntiles) {
        const RowTile rt = tile_info(cc);
        if (!hidden(rt)) {
          const Ops o = front(tc, rt, cc.buf);
          if constexpr (DEFER) {
            pend_ops = o;
            pend_buf = cc.buf;
            pend = true;
          } else {
            back(cc.buf, o);
          }
        }
        advance(cc);
      }
      if (dq_on) {
        // the dS-waves published tile t - 2 one barrier ago
        const int tq = t - 2;
        if (tq >= 0 && tq < ntiles) {
          dq_step(tq, tile_info(cq));
          advance(cq);
        }
      }
      tile_barrier();
    }
    // a dS-wave's last tile (its buffer is no longer reloaded)
    if constexpr (DEFER) {
      if (pend) back(pend_buf, pend_ops);
    }
  };
  if (NP > 2 && defer)
    sweep(StepOrder<true>{});
  else
    sweep(StepOrder<false>{});

  // ---- epilogue: acc[db][i] is dV^T or dK^T at d = 32 db + c_row0(i) + 4 h,
  // key wave_k0 + r
  if (wave_k0 + r >= kseg) return;
  const int key = wave_k0 + r;
  const float sc = pw ? 1.f : a.scale;
  if (R > 1) {
    // this share's scaled partial; bwd_kv_combine applies the epilogue
    const size_t krow = kpre ? (size_t)key : (size_t)a.P + kbase + key;
    const size_t nrows = (size_t)a.P + a.total_len;
    float* part = (pw ? a.part_dv : a.part_dk) + (((size_t)rs * nrows + krow) * a.hkv + hk) * D + 4 * h;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        *(float4*)(part + 32 * db + 8 * g4) =
            make_float4(acc[db][4 * g4] * sc, acc[db][4 * g4 + 1] * sc, acc[db][4 * g4 + 2] * sc,
                        acc[db][4 * g4 + 3] * sc);
    return;
  }
  if (kpre) {
    const size_t off = ((size_t)key * a.hkv + hk) * D + 4 * h;
    float* cache = pw ? a.gv : a.gk;
    // every cache value is loaded before the first store, so the loads are
    // in flight together instead of one round trip each
    float4 cv[NDB][4];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) cv[db][g4] = *(const float4*)(cache + off + 32 * db + 8 * g4);
    if (a.pk_mode == kPkAccumulate) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          float4 c = cv[db][g4];
          c.x += acc[db][4 * g4] * sc;
          c.y += acc[db][4 * g4 + 1] * sc;
          c.z += acc[db][4 * g4 + 2] * sc;
          c.w += acc[db][4 * g4 + 3] * sc;
          *(float4*)(cache + off + 32 * db + 8 * g4) = c;
        }
    } else {
      bf16* out = (bf16*)(pw ? a.dv_p : a.dk_p);
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const float4 c = cv[db][g4];
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
  int tile, z, hq, split;
};
__device__ __forceinline__ QBlock decode_q_block(const AttnArgs& a, int bid, int ntx) {
  const int G = a.hq / a.hkv;
  int b = bid;
  const int hk = b % a.hkv;
  b /= a.hkv;
  const int gi = b % G;
  b /= G;
  QBlock qb;
  qb.split = b % a.n_split;
  b /= a.n_split;
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
    const SegRows sg = suffix_rows(a.cu, seq, a.total_len);
    row_base = sg.base;
    seg_len = sg.len;
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
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      settle(qf[s]);
      settle(df[s]);
    }
    settle(lse2);
    settle(drow);
  }
  f32x16 dq[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) dq[db] = zero16();

  const int last_lp = min(lp0 + kQBQ, seg_len) - 1;
  const int nkeys0 = prefix_rows ? min(a.P, last_lp + 1) : a.P;
  const int nkeys1 = prefix_rows ? 0 : last_lp + 1;
  const int nt0 = (nkeys0 + BK - 1) / BK, nt1 = (nkeys1 + BK - 1) / BK;
  // this split's share [t_begin, t_end) of the nt0 + nt1 key tiles
  const int t_begin = (int)((long)(nt0 + nt1) * blk.split / a.n_split);
  const int t_end = (int)((long)(nt0 + nt1) * (blk.split + 1) / a.n_split);

  const bf16 *k_p = in_sgpr((const bf16*)a.k_p), *k_s = in_sgpr((const bf16*)a.k_s);
  const bf16 *v_p = in_sgpr((const bf16*)a.v_p), *v_s = in_sgpr((const bf16*)a.v_s);
  TileLoader<D, 4, BK> tl;
  tl.init(a.hkv, w, lane);
  auto issue = [&](int t, bf16* Kd, bf16* Vd) {
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

  if (!row_valid) return;
  // dq[db][i] = dQ^T[d = 32 db + c_row0(i) + 4 h][row my_lp] (unscaled)
  const size_t off = ((size_t)(row_base + my_lp) * a.hq + hq) * D + 4 * h;
  if (a.n_split > 1) {
    // suffix rows only: this split's partial, merged by bwd_dq_combine
    float* part = a.part_dq + (size_t)blk.split * a.total_len * a.hq * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        *(float4*)(part + off + 32 * db + 8 * g4) =
            make_float4(dq[db][4 * g4], dq[db][4 * g4 + 1], dq[db][4 * g4 + 2], dq[db][4 * g4 + 3]);
    return;
  }
  if (prefix_rows && a.dq_p_accumulate) {
    // dense baseline: the prefix rows' dQ sums over the trajectories (all
    // loads before the first store)
    float* acc = a.dq_acc_p;
    float4 cv[NDB][4];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) cv[db][g4] = *(const float4*)(acc + off + 32 * db + 8 * g4);
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        float4 v = cv[db][g4];
        v.x += dq[db][4 * g4];
        v.y += dq[db][4 * g4 + 1];
        v.z += dq[db][4 * g4 + 2];
        v.w += dq[db][4 * g4 + 3];
        *(float4*)(acc + off + 32 * db + 8 * g4) = v;
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
// so the XCD mapping of each role holds.  The atomic-dQ variant (AQ) has the
// key-outer role only: its blocks also add dQ into fp32 accumulators.
template <int D, bool AQ>
__global__ __launch_bounds__(kThreads, 2) void bwd_bf16_kernel(AttnArgs a, int n_first, int n_kv,
                                                               int n_q, int kv_first) {
  constexpr int TE = Tile<D>::ELEMS;
  // one LDS block shared by the two roles: the query-outer role's four
  // 64-key tiles, or the key-outer role's KvLds
  constexpr int kQBytes = AQ ? 0 : 4 * TE * 2;
  constexpr int kBytes = sizeof(KvLds<D, AQ>) > kQBytes ? sizeof(KvLds<D, AQ>) : kQBytes;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kBytes];
  const int b = blockIdx.x;
  if constexpr (AQ) {
    if (b < n_kv) bwd_kv_body<D, true>(a, b, *(KvLds<D, true>*)lds);
    return;
  } else {
    const bool first = b < n_first;
    const int bid = first ? b : b - n_first;
    // the first segment is padded to a multiple of 8 blocks: padding exits
    if (first == (kv_first != 0)) {
      if (bid < n_kv) bwd_kv_body<D, false>(a, bid, *(KvLds<D, false>*)lds);
    } else {
      bf16(*tiles)[TE] = (bf16(*)[TE])lds;
      if (bid < n_q) bwd_q_body<D>(a, bid, tiles, tiles + 2);
    }
  }
}

// The key-outer role alone, kKvWidePairs wave pairs (192 keys) per
// workgroup and one workgroup per CU: three waves on every SIMD, where the
// shared launch holds two (the query-outer role needs more registers than a
// third wave leaves; the key-outer role fits in 168).  Each wave's tile is a
// chain of dependent steps (LDS reads, a product, the elementwise step, the
// second product), so a third wave per SIMD fills more of the matrix core's
// idle cycles; the pairs also share each Q/dO tile load.  Twelve waves keep
// the SIMDs even (waves w, w + 4, w + 8 share one).
template <int D, bool PC>
__global__ __launch_bounds__(kKvWidePairs * 128, 1) void bwd_kv_wide_kernel(AttnArgs a, int n_kv) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[sizeof(KvLds<D, false, kKvWidePairs>)];
  if ((int)blockIdx.x < n_kv)
    bwd_kv_body<D, false, kKvWidePairs, PC>(a, blockIdx.x, *(KvLds<D, false, kKvWidePairs>*)lds);
}

// dQ of every (suffix row, q head) = scale * the sum of the n_split partials
// in split order.  One group of D / 4 threads per (row, head), 16-byte reads.
template <int D>
__global__ __launch_bounds__(256) void bwd_dq_combine_kernel(AttnArgs a) {
  constexpr int TPR = D / 4;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const long rh = idx / TPR;  // row * hq + head
  const int c = (int)(idx % TPR);
  const long nrh = (long)a.total_len * a.hq;
  if (rh >= nrh) return;
  float4 acc = *(const float4*)(a.part_dq + rh * D + 4 * c);
  for (int j = 1; j < a.n_split; ++j) {
    const float4 v = *(const float4*)(a.part_dq + ((size_t)j * nrh + rh) * D + 4 * c);
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  const bf16x4 o = {(bf16)(acc.x * a.scale), (bf16)(acc.y * a.scale), (bf16)(acc.z * a.scale),
                    (bf16)(acc.w * a.scale)};
  *(bf16x4*)((bf16*)a.dq_s + rh * D + 4 * c) = o;
}

// dK/dV of every key of a launch whose key-outer role split its row sweeps:
// the kv_rsplit partials summed in share order, then the launch's epilogue
// (prefix keys: cache += sum, or storage = sum + cache; suffix keys:
// storage = sum).  Keys: the n_pre prefix keys, then the packed rows
// cu[seq_base] .. cu[seq_base + n_seq] - 1 (at most n_sfx of them).  One
// group of D / 4 threads per (key, kv head), 16-byte accesses.
template <int D>
__global__ __launch_bounds__(256) void bwd_kv_combine_kernel(AttnArgs a, int n_pre, int n_sfx) {
  constexpr int TPR = D / 4;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const long kh = idx / TPR;  // (key index) * hkv + kv head
  const int c = (int)(idx % TPR);
  const long n_pre_kh = (long)n_pre * a.hkv;
  if (kh >= n_pre_kh + (long)n_sfx * a.hkv) return;
  const bool pre = kh < n_pre_kh;
  const int hk = (int)(kh % a.hkv);
  long key;
  if (pre) {
    key = kh / a.hkv;
  } else {
    const SegRows sp = suffix_span(a.cu, a.seq_base, a.seq_base + a.n_seq, a.total_len);
    const int r0 = sp.base, r1 = sp.base + sp.len;
    key = r0 + (kh - n_pre_kh) / a.hkv;
    if (key >= r1) return;
  }
  const size_t nrows = (size_t)a.P + a.total_len;
  const size_t krow = pre ? (size_t)key : (size_t)a.P + key;
  const size_t off = (krow * a.hkv + hk) * D + 4 * c;
  const size_t stride = nrows * a.hkv * D;
  float4 sk = *(const float4*)(a.part_dk + off), sv = *(const float4*)(a.part_dv + off);
  for (int j = 1; j < a.kv_rsplit; ++j) {
    const float4 k4 = *(const float4*)(a.part_dk + j * stride + off);
    const float4 v4 = *(const float4*)(a.part_dv + j * stride + off);
    sk.x += k4.x; sk.y += k4.y; sk.z += k4.z; sk.w += k4.w;
    sv.x += v4.x; sv.y += v4.y; sv.z += v4.z; sv.w += v4.w;
  }
  const size_t o = ((size_t)key * a.hkv + hk) * D + 4 * c;
  if (pre) {
    float4* gk = (float4*)(a.gk + o);
    float4* gv = (float4*)(a.gv + o);
    const float4 ck = *gk, cv = *gv;
    if (a.pk_mode == kPkAccumulate) {
      *gk = make_float4(ck.x + sk.x, ck.y + sk.y, ck.z + sk.z, ck.w + sk.w);
      *gv = make_float4(cv.x + sv.x, cv.y + sv.y, cv.z + sv.z, cv.w + sv.w);
    } else {
      *(bf16x4*)((bf16*)a.dk_p + o) = bf16x4{(bf16)(sk.x + ck.x), (bf16)(sk.y + ck.y),
                                             (bf16)(sk.z + ck.z), (bf16)(sk.w + ck.w)};
      *(bf16x4*)((bf16*)a.dv_p + o) = bf16x4{(bf16)(sv.x + cv.x), (bf16)(sv.y + cv.y),
                                             (bf16)(sv.z + cv.z), (bf16)(sv.w + cv.w)};
    }
  } else {
    *(bf16x4*)((bf16*)a.dk_s + o) = bf16x4{(bf16)sk.x, (bf16)sk.y, (bf16)sk.z, (bf16)sk.w};
    *(bf16x4*)((bf16*)a.dv_s + o) = bf16x4{(bf16)sv.x, (bf16)sv.y, (bf16)sv.z, (bf16)sv.w};
  }
}

namespace {
// the row shares' partial dK/dV summed in share order, with the epilogue
hipError_t launch_kv_combine(const AttnArgs& a, int head_dim, hipStream_t st) {
  const int n_pre = a.n_prefix_k_tiles > 0 ? a.P : 0;
  const int n_sfx = a.n_seq * a.n_suffix_k_tiles > 0 ? a.total_len : 0;
  const long kthreads = ((long)n_pre + n_sfx) * a.hkv * (head_dim / 4);
  const unsigned kb = (unsigned)((kthreads + 255) / 256);
  ProfileScope pk("bwd_kv_combine", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(bwd_kv_combine_kernel<64>, dim3(kb), dim3(256), 0, st, a, n_pre, n_sfx);
  else
    hipLaunchKernelGGL(bwd_kv_combine_kernel<128>, dim3(kb), dim3(256), 0, st, a, n_pre, n_sfx);
  return hipGetLastError();
}
}  // namespace

int bwd_bf16_kv_wide_block_k() { return 32 * kKvWidePairs; }
int bwd_bf16_kv_wide_slots() { return 256; }  // one workgroup per CU

hipError_t launch_bwd_bf16_kv_wide(const AttnArgs& a, int head_dim, hipStream_t st) {
  // key-outer blocks only, 32 * kKvWidePairs-key tiles, default (non-atomic) mode
  if (a.dq_atomic || a.n_prefix_q_tiles || a.n_suffix_q_tiles || a.n_split > 1)
    return hipErrorInvalidValue;
  const int R = a.kv_rsplit > 1 ? a.kv_rsplit : 1;
  if (R > 1 && (a.part_dk == nullptr || a.part_dv == nullptr)) return hipErrorInvalidValue;
  const long n_kt = (long)a.n_prefix_k_tiles + (long)a.n_seq * a.n_suffix_k_tiles;
  const long n_kv = n_kt * a.hkv * R;
  if (n_kv == 0) return hipSuccess;
  {
    ProfileScope ps("bwd_bf16", st);
    // Phase C: prefix key tiles and causal prefix rows only
    const bool pc = a.prefix_rows && !a.suffix_rows && a.n_seq * a.n_suffix_k_tiles == 0;
    const dim3 grid((unsigned)n_kv), block(kKvWidePairs * 128);
    if (head_dim == 64) {
      if (pc)
        hipLaunchKernelGGL((bwd_kv_wide_kernel<64, true>), grid, block, 0, st, a, (int)n_kv);
      else
        hipLaunchKernelGGL((bwd_kv_wide_kernel<64, false>), grid, block, 0, st, a, (int)n_kv);
    } else if (pc) {
      hipLaunchKernelGGL((bwd_kv_wide_kernel<128, true>), grid, block, 0, st, a, (int)n_kv);
    } else {
      hipLaunchKernelGGL((bwd_kv_wide_kernel<128, false>), grid, block, 0, st, a, (int)n_kv);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return R > 1 ? launch_kv_combine(a, head_dim, st) : hipSuccess;
}

hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, int n_qz, bool deterministic,
                           hipStream_t st) {
  if (a.n_split > 1 && (a.prefix_rows || a.part_dq == nullptr)) return hipErrorInvalidValue;
  const int R = a.kv_rsplit > 1 ? a.kv_rsplit : 1;
  if (R > 1 && (a.part_dk == nullptr || a.part_dv == nullptr)) return hipErrorInvalidValue;
  // the atomic-dQ launch has no query-outer role, and needs an accumulator
  // for every kind of row its key tiles sweep
  (void)deterministic;  // the default path has no atomics; the atomic one is asked for explicitly
  const bool aq = a.dq_atomic != 0;
  if (aq && (a.n_prefix_q_tiles || a.n_suffix_q_tiles || a.n_split > 1 ||
             (a.prefix_rows && a.dq_acc_p == nullptr) || (a.n_seq > 0 && a.dq_acc_s == nullptr)))
    return hipErrorInvalidValue;
  const long n_kt = (long)a.n_prefix_k_tiles + (long)a.n_seq * a.n_suffix_k_tiles;
  const long n_kv = n_kt * a.hkv * R;
  const long n_q = (long)(a.n_prefix_q_tiles + a.n_suffix_q_tiles) * a.hq * n_qz * a.n_split;
  if (n_kv + n_q == 0) return hipSuccess;
  // Which role's blocks start first.  Phase C / dense prefix: the key-outer
  // role, whose causal key tile 0 sweeps every prefix row.  Phase B: the
  // query-outer role only when its blocks are much longer (by over 2.5x),
  // so that they do not start last and end the launch on a tail; where the
  // lengths are close, the key-outer role (the one with more blocks) leads
  // and the query-outer blocks fill the slots its last round leaves.  The
  // longest key-outer block sweeps the G heads of every row of the launch (a
  // prefix key tile sees all of them; without a prefix, a suffix key tile
  // sees its own), cut into R shares; the longest query-outer block visits
  // all prefix key tiles and its own suffix's, cut into n_split ranges.  A
  // query-outer step (128 rows x 64 keys, three products) costs about two
  // key-outer steps (32 rows x 64 keys, four products).
  int kv_first = 1;
  if (!aq && !a.prefix_rows && n_q > 0) {
    const long rows = a.n_prefix_k_tiles > 0 ? a.total_len : (long)a.n_suffix_k_tiles * kKvBK;
    const long kv_len = (long)(a.hq / a.hkv) * ((rows + 31) / 32) / R;
    const long nkt = (long)a.n_prefix_k_tiles + a.n_suffix_k_tiles;
    const long ns = a.n_split > 1 ? a.n_split : 1;
    const long q_len = 2 * ((nkt + ns - 1) / ns);
    kv_first = 2 * q_len > 5 * kv_len ? 0 : 1;
  }
  const long first = kv_first ? n_kv : n_q;
  const long n_first = aq ? n_kv : (first + 7) / 8 * 8;
  const long nb = n_first + (kv_first ? n_q : n_kv);
  ProfileScope ps("bwd_bf16", st);
  if (aq) {
    if (head_dim == 64)
      hipLaunchKernelGGL((bwd_bf16_kernel<64, true>), dim3((unsigned)nb), dim3(kThreads), 0, st, a,
                         (int)n_first, (int)n_kv, 0, 1);
    else
      hipLaunchKernelGGL((bwd_bf16_kernel<128, true>), dim3((unsigned)nb), dim3(kThreads), 0, st, a,
                         (int)n_first, (int)n_kv, 0, 1);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL((bwd_bf16_kernel<64, false>), dim3((unsigned)nb), dim3(kThreads), 0, st, a,
                       (int)n_first, (int)n_kv, (int)n_q, kv_first);
  } else {
    hipLaunchKernelGGL((bwd_bf16_kernel<128, false>), dim3((unsigned)nb), dim3(kThreads), 0, st, a,
                       (int)n_first, (int)n_kv, (int)n_q, kv_first);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (R > 1 && n_kt > 0 && (e = launch_kv_combine(a, head_dim, st)) != hipSuccess) return e;
  if (a.n_split <= 1) return hipSuccess;
  const long threads = (long)a.total_len * a.hq * (head_dim / 4);
  const unsigned cb = (unsigned)((threads + 255) / 256);
  ProfileScope pc("bwd_dq_combine", st);
  if (head_dim == 64)
    hipLaunchKernelGGL(bwd_dq_combine_kernel<64>, dim3(cb), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(bwd_dq_combine_kernel<128>, dim3(cb), dim3(256), 0, st, a);
  return hipGetLastError();
}

int bwd_bf16_block_q() { return kQBQ; }

int bwd_bf16_kvsplit(long kv_tiles, long max_tiles, bool kv_alone, int slots) {
  // kv_tiles: the key-outer role's (32-row tile, q head) steps over all its
  // blocks; max_tiles: the longest block's.  The query-outer role adds about
  // 3/4 of that work (three products per visible block instead of four),
  // spread over `slots` workgroup slots (two per CU on 256 CUs, one for
  // the key-outer-only launch); kv_alone: the launch has no
  // query-outer role (atomic dQ, whose dQ product lengthens every step
  // alike, or the key-outer-only launch).  A
  // block clearly longer than that average per slot (by over 10%: the
  // shares' partials and combine cost about that much) would end the launch
  // alone: then every key tile's sweep is cut into R contiguous shares,
  // about the average each, at most 8 and at least 16 steps each.
  if (kv_tiles <= 0 || max_tiles <= 0) return 1;
  const double per_slot = (kv_alone ? 1.0 : 1.75) * (double)kv_tiles / (double)slots;
  if ((double)max_tiles <= 1.1 * per_slot) return 1;
  long r = (long)std::ceil((double)max_tiles / per_slot);
  r = std::min(r, max_tiles / 16);
  return (int)std::max(1L, std::min(r, 8L));
}

int bwd_bf16_qsplit(int n_row_blocks, int n_key_tiles) {
  // Only when the query-outer blocks alone cannot fill two slots per CU on
  // 256 CUs; each split keeps at least 16 key tiles, so that a split costs
  // about half of a key-outer block and packs into the tail of the launch.
  if (n_row_blocks <= 0 || n_row_blocks >= 512) return 1;
  int ns = std::min(n_key_tiles / 16, (512 + n_row_blocks - 1) / n_row_blocks);
  return std::max(1, std::min(ns, 8));
}

}  // namespace spr
