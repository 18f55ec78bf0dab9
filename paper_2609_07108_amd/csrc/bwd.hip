// Backward branch attention for one context-parallel rank share (Sec. 3.2:
// the gradients walk the KV ring a second time and each rank sums its
// contributions where it is).
//
// With the final LSE of every row the probabilities of any key subset are
// P = exp(S - LSE), so the merge of Eq. lse-merge needs no explicit backward:
// every ring-step block and the branch-local keys contribute
//   dV += P^T dO,  dS = P o (dP - Delta),  dP = dO V^T,  Delta = <dO, O>,
//   dK += scale dS^T Q,  dQ += scale dS K.
//
// Kernels
//   preprocess : -Delta and -LSE * log2(e) per (query token, head).
//   kv         : dK and dV.  One workgroup per 128 keys of one ring-step
//                block, sequence and KV head, as two wavefront pairs of 64
//                keys (one wavefront of a pair computes P and dV, the other
//                dS and dK, with P handed over in LDS); it walks the query
//                tokens that reach those keys in 64-row tiles (tokens x the
//                G heads of the KV head), prefetched into LDS by direct
//                global-to-LDS loads.  No atomics.
//   dq         : dQ, query-tile parallel like the forward (256-row tiles,
//                64 rows per wavefront): per key tile S^T = K Q^T,
//                dP^T = V dO^T, dS^T, dQ^T += K^T dS^T, software-pipelined
//                across key tiles; the branch-local keys' terms are the
//                accumulators' start value in the fused schedule (from the
//                tile's branch keys staged once in LDS) and are added by the
//                finalize kernel in the per-step one.
//                Splitting dQ off
//                costs two extra contractions but avoids fp32 atomics, whose
//                throughput (about one 4-byte update per L2 channel and clock)
//                would otherwise bound the whole backward.
//   branch     : dK and dV of the branch-local keys (at most 64 per group).
#include <type_traits>

#include "ba_internal.h"
#include "device_common.h"
#include "kernels.h"

namespace ba {

namespace {

__device__ __forceinline__ const bf16* row_ptr(const bf16* main, const bf16* br, int32_t qrow,
                                               int32_t hq, int32_t head) {
  return qrow >= 0 ? main + ((int64_t)qrow * hq + head) * kHeadDim
                   : br + ((int64_t)(-qrow - 1) * hq + head) * kHeadDim;
}

__device__ __forceinline__ void store_grad(void* base, int64_t idx, float v, bool f32) {
  if (f32) static_cast<float*>(base)[idx] = v;
  else static_cast<bf16*>(base)[idx] = (bf16)v;
}

// Operand fragments of a 64-row plane tile sit at compile-time offsets from
// four per-lane bases: row fragments (rows 32 rb + qi, columns 16 c + 8h;
// the chunk permutation depends on c only through its parity) from
// row_even / row_odd, transposed fragments (rows 16 t + 4h + {0..3} and
// 16 t + 8 + 4h + {0..3}, columns 32 nt + ..) from tr_lo / tr_hi.  A
// tile's bases (LDS byte addresses) are made opaque to the compiler, which
// would otherwise re-associate the constant offsets into one register per
// fragment.
constexpr int kOpRows = 64;
static_assert(kBwdRows == kOpRows && kFwdKeys == kOpRows, "operand tiles are 64 rows");
struct LaneOffsets {
  int row_even, row_odd, tr_lo, tr_hi;
};
__device__ __forceinline__ LaneOffsets lane_offsets(int lane) {
  const int qi = lane & 31, half = lane >> 5, trc = (lane & 16) + 4 * (lane & 3);
  return LaneOffsets{tile_off<kOpRows>(qi, 8 * half), tile_off<kOpRows>(qi, 16 + 8 * half),
                     tile_off<kOpRows>(4 * half + ((lane & 15) >> 2), trc),
                     tile_off<kOpRows>(8 + 4 * half + ((lane & 15) >> 2), trc)};
}
struct OpBases {
  uint32_t re, ro, tl, th;
};
// row fragments of rowT, transposed fragments of trT
__device__ __forceinline__ OpBases op_bases(const LaneOffsets& l, const bf16* rowT, const bf16* trT) {
  OpBases o{lds_lane_addr(rowT + l.row_even), lds_lane_addr(rowT + l.row_odd), lds_lane_addr(trT + l.tr_lo),
            lds_lane_addr(trT + l.tr_hi)};
  asm volatile("" : "+v"(o.re), "+v"(o.ro), "+v"(o.tl), "+v"(o.th));
  return o;
}
__device__ __forceinline__ bf16x8 row_frag(const OpBases& o, int rb, int c) {
  return lds_ld16(((c & 1) ? o.ro : o.re) + (uint32_t)(((c >> 1) * kOpRows + 32 * rb) * 64));
}
__device__ __forceinline__ bf16x8 tr_frag(const OpBases& o, int t, int nt) {
  const uint32_t off = (uint32_t)((nt * kOpRows + 16 * t) * 64);
  const bf16x4 lo = lds_ld_tr4(o.tl + off), hi = lds_ld_tr4(o.th + off);
  return bf16x8(__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

}  // namespace

// ------------------------------------------------------------ preprocess
// 16 lanes (a DPP row) per (token, head), 16 bytes each: -Delta = -<dO, O>
// over 128 dims and -LSE in log2 units (both stored negated so the dK/dV
// kernel can start its S and dP accumulations from them); Q and dO rows are
// also copied into token order, so the dK/dV kernel addresses a query tile
// without indirection.  Rows past the end redo the last row and write
// nothing (the DPP row sum needs every lane).
__global__ __launch_bounds__(256) void bwd_preprocess_kernel(BwdParams p) {
  const int64_t rows = (int64_t)p.num_tokens * p.hq;
  const int64_t pair0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
  const bool live = pair0 < rows;
  const int64_t pair = live ? pair0 : rows - 1;
  const int sub = threadIdx.x & 15;
  const int32_t t = (int32_t)(pair / p.hq);
  const int32_t head = (int32_t)(pair - (int64_t)t * p.hq);
  const TokInfo tk = p.toks[t];
  const bf16x8 ov = ld16(row_ptr(p.o_main, p.o_br, tk.qrow, p.hq, head) + 8 * sub);
  const bf16x8 gv = ld16(row_ptr(p.do_main, p.do_br, tk.qrow, p.hq, head) + 8 * sub);
  const bf16x8 qv = ld16(row_ptr(p.q_main, p.q_br, tk.qrow, p.hq, head) + 8 * sub);
  float dlt = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) dlt += (float)ov[e] * (float)gv[e];
  dlt = row16_sum(dlt);
  if (!live) return;
  st16(p.qtok + pair * kHeadDim + 8 * sub, qv);
  st16(p.gtok + pair * kHeadDim + 8 * sub, gv);
  if (sub == 0) {
    const float lse = tk.qrow >= 0 ? p.lse_main[(int64_t)head * p.n_local + tk.qrow]
                                   : p.lse_br[(int64_t)head * p.n_br + (-tk.qrow - 1)];
    p.rowstat[pair] = make_float2(-lse * kLog2e, -dlt);
  }
}

// ------------------------------------------------------------ kv (ring)
// Workgroup of 4 wavefronts (one per SIMD, up to 512 registers each) on 128
// keys, as two wavefront pairs of 64 keys: pair p owns keys 64p..64p+63.
// Inside a pair the work of the four contractions is split by operand:
//   score wavefront (w = p):     K of the pair's keys in registers;
//                                S = Q K^T, P = exp2(S scale log2e - LSE
//                                log2e) with the causal mask (one fused
//                                multiply-add and one exp2 per element), P
//                                handed to the partner through LDS,
//                                dV += P^T dO
//   gradient wavefront (w = 2+p): V in registers; dP - Delta = dO V^T -
//                                Delta (the accumulation starts from
//                                -Delta), dS = P o (dP - Delta) with P read
//                                back, dK += dS^T Q
// Each wavefront runs 64 MFMAs per 64-row query tile and every Q or dO
// operand fragment it reads from LDS feeds two of them (the pair's two
// 32-key blocks), so the operand traffic per MFMA is half that of a
// wavefront on 32 keys; the dK and dV accumulators of 64 keys (256
// registers) sit in two register files.  No atomics.
//
// Query tiles (tokens x the G heads of the KV head, ordered by causal limit)
// are walked from the last down or from the first up, as the planner sets
// per item (walk_down) so that items running at the same time read the
// same Q and dO tiles at about the same time and share them in L2.  Below,
// "tile i" of a stage is the one at stage position i.  In stage i the score wavefronts compute P of tile
// i+1 and dV of tile i (P of tile i kept in registers from stage i-1); the
// gradient wavefronts compute dK of tile i with P of tile i written by their
// partner in stage i-1.  One barrier per stage publishes P and the direct
// loads.  Q of tile k (with per-row LSE and causal limit) is read in stages
// k-1 and k and rotates through four LDS buffers; dO of tile k (with per-row
// -Delta) is read in stage k and rotates through three; both are loaded two
// stages before their first use by direct global-to-LDS loads, at addresses
// computed from the token index alone (token-ordered copies of Q and dO), so
// the loops have no compiler-visible memory loads and the waits on the loads
// are explicit.  Inside a stage the MFMAs, their operand reads, the softmax
// (or dS) elements and the P writes follow a fixed slot schedule.
namespace {

constexpr int kKvWaves = 4;
constexpr int kKvThreads = 64 * kKvWaves;
constexpr int kOpAhead = 2;  // operand fragments read ahead of their MFMAs (two MFMAs each)
constexpr int kQBufs = 4;
constexpr int kGBufs = 3;

struct QSide {
  bf16 q[kBwdRows * kHeadDim];
  float l2[kBwdRows];  // -LSE * log2 e
  int pl[kBwdRows];    // causal limit P (-1: no token)
};
struct GSide {
  bf16 g[kBwdRows * kHeadDim];
  float nd[kBwdRows];  // -Delta
};
struct KvLds {
  QSide qs[kQBufs];
  GSide gs[kGBufs];
  // P of a tile as MFMA operand fragments: [tile parity][pair][4 rb + 2 kb
  // + tt][lane] (rows 32 rb + 16 tt.., keys 32 kb.. of the pair)
  bf16x8 x[2][2][8][64];
};

// slot of softmax element e (score wavefront) and of dS element e (gradient
// wavefront) in a stage's 64-slot schedule
// (score elements start 7 slots after the last S MFMA of row block 0: the
// S MFMAs are inline assembly, so the compiler does not pad the 12 wait
// states between them and a vector read of their result)
constexpr int a_slot(int e) { return 22 + (e * 41) / 64; }
constexpr int b_slot(int e) { return 17 + (e * 38) / 64; }

}  // namespace

__global__ __launch_bounds__(kKvThreads, 1) void bwd_kv_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) KvLds sm;
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

  const BwdTile tile = p.tiles[blockIdx.x];
  const SeqInfo seq = p.seqs[tile.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wavefront-uniform
  const int qi = lane & 31;
  const int half = lane >> 5;
  const bool scorer = wave < 2;
  const int pair = wave & 1;
  const int G = p.G;
  const int tpt = kBwdRows / G;  // tokens per query tile
  const int ntiles = (tile.q_end - tile.q_begin + tpt - 1) / tpt;  // >= 1 (planner)
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  const int64_t key0 = (int64_t)seq.seg_off + tile.u0;  // first key row in the block
  const int head0 = tile.kvh * G;

  // ---- the lane's keys 64 pair + 32 kb + qi: the position decides
  // visibility (visible to a row iff position <= the row's causal limit;
  // local index < c lies in chunk `step`, the rest in chunk 2C-1-step)
  int kpos[2], kload[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int my_key = 64 * pair + 32 * kb + qi;
    kload[kb] = my_key < tile.nk ? my_key : tile.nk - 1;
    const int u = tile.u0 + my_key;
    kpos[kb] = u < seq.c ? tile.step * seq.c + u : (2 * p.C - 1 - tile.step) * seq.c + (u - seq.c);
    if (my_key >= tile.nk) kpos[kb] = 0x7fffffff;
  }

  // ---- direct loads: the score wavefronts load Q rows 32 w + 16 j + lane/4
  // (j = 0, 1), the gradient wavefronts the same rows of dO; wavefront 0
  // also loads the tile's LSE, 1 its causal limits, 2 and 3 its -Delta.  Rows
  // without a token read the tile's first row (finite data) and the
  // sentinel token's limit -1.
  int dtl[2], dhg[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = 32 * pair + 16 * j + (lane >> 2);
    dtl[j] = row / G;
    dhg[j] = row - dtl[j] * G;
  }
  const int stl = lane / G, shg = lane - stl * G;
  const uint32_t q_lds = lds_addr(&sm.qs[0]);
  const uint32_t g_lds = lds_addr(&sm.gs[0]);
  // Q of the tile at stage position kq (score wavefronts) or dO of the one
  // at position kg (gradient wavefronts); past the last position its tile
  // again, into the position's own (idle) buffer.  A stage's loads go out in 9 pieces in its first slots (the
  // buffers they fill, those of tile s-1, are free from the stage's start):
  // pieces 0-7 are the row loads (rows 32 pair + 16 (piece/4) + lane/4,
  // plane piece%4), piece 8 the statistic.
  const bf16* rows_src = scorer ? p.qtok : p.gtok;
  asm volatile("" : "+s"(rows_src));  // kept in registers, not re-read per stage
  struct DmaStage {
    int qt0, nt;
    uint32_t b;
  };
  // the query tile at stage position k (see walk_down)
  auto tile_at = [&](int k) { return tile.walk_down ? ntiles - 1 - k : k; };
  auto dma_begin = [&](int kq, int kg) __attribute__((always_inline)) {
    const int k = scorer ? kq : kg;
    DmaStage d;
    d.qt0 = tile.q_begin + tile_at(k < ntiles ? k : ntiles - 1) * tpt;
    d.nt = tile.q_end - d.qt0;  // tokens left from qt0
    d.b = scorer ? q_lds + (uint32_t)(k % kQBufs) * (uint32_t)sizeof(QSide)
                 : g_lds + (uint32_t)(k % kGBufs) * (uint32_t)sizeof(GSide);
    return d;
  };
  auto dma_piece = [&](const DmaStage& d, int piece) __attribute__((always_inline)) {
    if (piece == 8) {
      // one statistic per wavefront, chosen by wavefront-uniform selects
      // (no branch between the first MFMA slots); wavefront 3 repeats
      // wavefront 2's load (the same words into the same LDS buffer), so
      // every wavefront has nine loads per stage
      const bool ok = stl < tpt && stl < d.nt;
      const bool limits = wave == 1;
      const void* b_lim = uniform_ptr(p.toks + d.qt0);
      const void* b_stat = uniform_ptr(p.rowstat + (int64_t)d.qt0 * p.hq + head0);
      asm volatile("" : "+s"(b_lim), "+s"(b_stat));  // both computed: a select, not a branch
      const void* base = limits ? b_lim : b_stat;
      const int off_lim = (ok ? stl : p.num_tokens - d.qt0) * (int)sizeof(TokInfo) + (int)offsetof(TokInfo, P);
      const int off_stat = (ok ? stl * p.hq + shg : 0) * (int)sizeof(float2) + (wave == 0 ? 0 : 4);
      const uint32_t dst = wave == 0 ? (uint32_t)offsetof(QSide, l2)
                           : limits  ? (uint32_t)offsetof(QSide, pl)
                                     : (uint32_t)offsetof(GSide, nd);
      dma4_async(base, (uint32_t)(limits ? off_lim : off_stat), d.b + dst);
      return;
    }
    const int j = piece >> 2, pl = piece & 3;
    const void* base = uniform_ptr(rows_src + ((int64_t)d.qt0 * p.hq + head0) * kHeadDim);
    const bool okr = dtl[j] < tpt && dtl[j] < d.nt;
    const int r = okr ? dtl[j] * p.hq + dhg[j] : 0;  // row relative to (qt0, head0)
    const int m = 8 * pair + 4 * j + pl;
    const uint32_t off = (uint32_t)(r * kHeadDim + dma_col<kBwdRows>(m, lane)) * (uint32_t)sizeof(bf16);
    dma16_async(base, off, d.b + dma_dst_bytes<kBwdRows>(m));  // q and g open both sides
  };
  auto issue_all = [&](int kq, int kg) __attribute__((always_inline)) {
    const DmaStage d = dma_begin(kq, kg);
#pragma unroll
    for (int piece = 0; piece < 9; ++piece) dma_piece(d, piece);
  };
  // End of a stage: this wavefront's loads issued before the stage (the
  // tiles the next stage reads) have landed and its P writes are done; the
  // nine loads of this stage stay in flight.  The barrier publishes
  // everything to the workgroup.
  auto stage_end = [&]() __attribute__((always_inline)) {
    wait_vmcnt_lgkm0<9>();
    lds_barrier();
  };

  const LaneOffsets lo = lane_offsets(lane);

  // Tiles u_lo .. u_hi-1 need no mask: every row has a token and sees all
  // keys of the block (tokens from q_full on do).  Stage positions [t_lo,
  // t_hi) hold them.
  int t_lo = ntiles, t_hi = ntiles;
  if (tile.nk == kBwdKeys && tpt * G == kBwdRows) {
    const int u_lo = min(ntiles, max(0, (tile.q_full - tile.q_begin + tpt - 1) / tpt));
    const int u_hi = max(u_lo, (tile.q_end - tile.q_begin) / tpt);
    t_lo = tile.walk_down ? ntiles - u_hi : u_lo;
    t_hi = tile.walk_down ? ntiles - u_lo : u_hi;
  }

  // Q of tiles 0 and 1, dO of tile 0
  issue_all(0, 0);
  if (scorer) issue_all(1, 0);
  f32x16 acc[2][4];  // dV (score) or dK (gradient): [kb][d block], rows = keys, lane = dim
  auto zero_acc = [&]() {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) mfma32_acc_zero(acc[kb][nt]);
  };
  const bf16* kvsrc = (scorer ? p.k_step[tile.step] : p.v_step[tile.step]) + tile.kvh * kHeadDim;

  if (scorer) {
    // K of the lane's keys (B operands of S), resident in the accumulation
    // registers.  The softmax scale is applied in fp32 per score: folding it
    // into a bf16 copy of K perturbs every score by about 2^-9 of its
    // magnitude, which grows with the logits (dK, dV relative error 3e-2 at
    // score standard deviation 16 against 3e-3 at 1).
    bf16x8 kreg[2][8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const bf16x8 kr = ld16(kvsrc + (key0 + kload[kb]) * kv_row_stride + 16 * c + 8 * half);
        asm volatile("" : "=a"(kreg[kb][c]) : "0"(kr));
      }
    zero_acc();
    __builtin_amdgcn_s_waitcnt(0);
    lds_barrier();
    // ---------------------------------------------------------- score side
    // stage: S and P of the next tile (Q, LSE, limits in qn; P fragments
    // out to pn and to the exchange slot xw), dV of the current tile (dO in
    // gc, its P in pc).  MFMA j: j < 32 -> S[rb][kb] chunk c (rb = j/16,
    // c = (j/2)%8, kb = j%2); j >= 32 -> dV[kb][nt] with rows 16t.. (t =
    // (j-32)/8, nt = ((j-32)/2)%4, kb = j%2).  Operand fragment j/2 feeds
    // MFMAs j and j+1.
    typedef u32x4 PFrags[2][2][2];  // P as bf16 pairs: [rb][kb][tt]
    auto stage = [&](const QSide& qn, const GSide& gc, const PFrags& pc, PFrags& pn, bf16x8* xw, const DmaStage& dm,
                     auto mask_tag, auto next_tag, auto cur_tag) __attribute__((always_inline)) {
      constexpr bool MASK = decltype(mask_tag)::value;
      constexpr bool NEXT = decltype(next_tag)::value;
      constexpr bool CUR = decltype(cur_tag)::value;
      constexpr int f_lo = NEXT ? 0 : 16, f_hi = CUR ? 32 : 16;
      f32x16 s[2][2], nl[2];
      bf16x8 opq[kOpAhead + 1];
      int4 sp[2][4];
      float prv = 0.f;

      const OpBases ob = op_bases(lo, qn.q, gc.g);
      auto load_op = [&](int f) -> bf16x8 {
        if (f < 16) return row_frag(ob, f >> 3, f & 7);
        // rows 16t+4h+{0..3}, 16t+8+4h+{0..3}: the rows of the lane's P values
        return tr_frag(ob, (f - 16) >> 2, (f - 16) & 3);
      };
      auto load_nl = [&](int rb) {  // -LSE log2e of the accumulator rows of row block rb
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 l4 = *reinterpret_cast<const float4*>(&qn.l2[32 * rb + 8 * q + 4 * half]);
          nl[rb][4 * q] = l4.x;
          nl[rb][4 * q + 1] = l4.y;
          nl[rb][4 * q + 2] = l4.z;
          nl[rb][4 * q + 3] = l4.w;
        }
      };
      auto load_lim = [&](int rb, int q) {
        sp[rb][q] = *reinterpret_cast<const int4*>(&qn.pl[32 * rb + 8 * q + 4 * half]);
      };
      // element e: rb = e/32, q = (e/8)%4, kb = (e/4)%2, accumulator slot
      // v = 4q + e%4 (row 32 rb + 8q + 4h + e%4)
      auto element = [&](int e) {
        const int rb = e >> 5, q = (e >> 3) & 3, kb = (e >> 2) & 1, c = e & 3, v = 4 * q + c;
        float pr = fast_exp2(__builtin_fmaf(s[rb][kb][v], p.scale_log2, nl[rb][v]));
        if (MASK) {
          const int lim = c == 0 ? sp[rb][q].x : c == 1 ? sp[rb][q].y : c == 2 ? sp[rb][q].z : sp[rb][q].w;
          pr = kpos[kb] <= lim ? pr : 0.f;
        }
        if (v & 1) pn[rb][kb][v >> 3][(v & 7) >> 1] = pack_bf16x2(prv, pr);
        else prv = pr;
      };
      auto mfma = [&](int j, const bf16x8& a) {
        if (j < 32) {
          const int rb = j >> 4, c = (j >> 1) & 7, kb = j & 1;
          if (c == 0) mfma32_v_first(s[rb][kb], a, kreg[kb][0]);
          else mfma32_v(s[rb][kb], a, kreg[kb][c]);
        } else {
          const int jj = j - 32, t = jj >> 3, nt = (jj >> 1) & 3, kb = jj & 1;
          mfma32_acc<false>(acc[kb][nt], __builtin_bit_cast(bf16x8, pc[t >> 1][kb][t & 1]), a);  // P from the last stage
        }
      };

      if constexpr (NEXT) load_nl(0);
      static_for<kOpAhead>([&](auto ic) {
        constexpr int f = f_lo + decltype(ic)::value;
        if constexpr (f < f_hi) opq[f % (kOpAhead + 1)] = load_op(f);
      });
      static_for<64>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        constexpr int f = j >> 1;
        constexpr bool active = f >= f_lo && f < f_hi;
        if constexpr (active && (j & 1) == 0 && f + kOpAhead < f_hi)
          opq[(f + kOpAhead) % (kOpAhead + 1)] = load_op(f + kOpAhead);
        if constexpr (NEXT) {
          if constexpr (j == 6) load_nl(1);
          // causal limits of rows 32 rb + 8 q + 4h.. three slots before their elements
          if constexpr (MASK) {
            static_for<8>([&](auto gc_) {
              constexpr int g = decltype(gc_)::value;
              if constexpr (a_slot(8 * g) - 3 == j) load_lim(g >> 2, g & 3);
            });
          }
          static_for<64>([&](auto ec) {
            constexpr int e = decltype(ec)::value;
            if constexpr (a_slot(e) == j) element(e);
          });
          // a fragment (rows 32 rb + 16 tt.., keys 32 kb..) is complete with
          // its element of q = 2 tt + 1, c = 3
          static_for<8>([&](auto fc) {
            constexpr int fr = decltype(fc)::value;
            constexpr int rb = fr >> 2, kb = (fr >> 1) & 1, tt = fr & 1;
            if constexpr (a_slot(32 * rb + 8 * (2 * tt + 1) + 4 * kb + 3) + 1 == j)
              xw[fr * 64 + lane] = __builtin_bit_cast(bf16x8, pn[rb][kb][tt]);
          });
        }
        if constexpr (active) mfma(j, opq[f % (kOpAhead + 1)]);
        if constexpr (j == 2) dma_piece(dm, 8);
        if constexpr (j >= 3 && j < 11) dma_piece(dm, j - 3);
        __builtin_amdgcn_sched_barrier(0);
      });
    };

    PFrags pa, pb;  // P of the current tile in pa between stages
    int s = 0;
    // one stage s: P of tile s+1 (mask class given), dV of tile s
    auto one = [&](const PFrags& pc, PFrags& pn, auto mask_tag) __attribute__((always_inline)) {
      stage(sm.qs[(s + 1) % kQBufs], sm.gs[s % kGBufs], pc, pn, &sm.x[(s + 1) & 1][pair][0][0], dma_begin(s + 3, s + 2),
            mask_tag, std::true_type{}, std::true_type{});
      stage_end();
      ++s;
    };
    // stages [s, s_end), all of one mask class
    auto run = [&](int s_end, auto mask_tag) __attribute__((always_inline)) {
      while (s + 1 < s_end) {
        one(pa, pb, mask_tag);
        one(pb, pa, mask_tag);
      }
      if (s < s_end) {
        one(pa, pb, mask_tag);
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int tt = 0; tt < 2; ++tt) pa[rb][kb][tt] = pb[rb][kb][tt];
      }
      mfma_drain();  // accumulators settled before the compiler may move them
    };

    // stage -1: P of tile 0 only
    if (t_lo == 0 && t_hi > 0)
      stage(sm.qs[0], sm.gs[0], pb, pa, &sm.x[0][pair][0][0], dma_begin(2, 1), std::false_type{}, std::true_type{},
            std::false_type{});
    else
      stage(sm.qs[0], sm.gs[0], pb, pa, &sm.x[0][pair][0][0], dma_begin(2, 1), std::true_type{}, std::true_type{},
            std::false_type{});
    stage_end();
    // stages 0 .. ntiles-2 by the mask class of their next tile, then the last
    run(min(ntiles - 1, max(0, t_lo - 1)), std::true_type{});
    run(min(ntiles - 1, max(0, t_hi - 1)), std::false_type{});
    run(ntiles - 1, std::true_type{});
    stage(sm.qs[0], sm.gs[s % kGBufs], pa, pb, &sm.x[0][pair][0][0], dma_begin(s + 3, s + 2), std::true_type{},
          std::false_type{}, std::true_type{});
    stage_end();
    mfma_drain();
  } else {
    // ------------------------------------------------------- gradient side
    bf16x8 vreg[2][8];  // V of the lane's keys: B operands of dP = dO V^T
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int c = 0; c < 8; ++c) vreg[kb][c] = ld16(kvsrc + (key0 + kload[kb]) * kv_row_stride + 16 * c + 8 * half);
    zero_acc();
    __builtin_amdgcn_s_waitcnt(0);
    lds_barrier();

    // stage: dP - Delta and dS of the current tile (dO and -Delta in gc, P
    // from the exchange slot xr), dK with Q in qc.  MFMA j: j < 32 ->
    // dP[rb][kb] chunk c (as S on the score side); j >= 32 -> dK[kb][nt]
    // with rows 16t.. .  dS element e runs chunk-major: t = e/16 (rows
    // 16t.., accumulator slots 8 (t%2)..), kb = (e/8)%2, slot 8 (t%2) + e%8.
    auto stage = [&](const QSide& qc, const GSide& gc, const bf16x8* xr, const DmaStage& dm) __attribute__((always_inline)) {
      f32x16 dp[2][2], nd[2];
      bf16x8 opq[kOpAhead + 1];
      bf16x8 pf[2][2][2];  // P fragments [rb][kb][tt]
      u32x4 dsf[2][2][2];  // dS as bf16 pairs, the A operands of dK: [rb][kb][tt]
      float dsv = 0.f;

      const OpBases ob = op_bases(lo, gc.g, qc.q);
      auto load_op = [&](int f) -> bf16x8 {
        if (f < 16) return row_frag(ob, f >> 3, f & 7);
        return tr_frag(ob, (f - 16) >> 2, (f - 16) & 3);
      };
      auto load_nd = [&](int rb) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 d4 = *reinterpret_cast<const float4*>(&gc.nd[32 * rb + 8 * q + 4 * half]);
          nd[rb][4 * q] = d4.x;
          nd[rb][4 * q + 1] = d4.y;
          nd[rb][4 * q + 2] = d4.z;
          nd[rb][4 * q + 3] = d4.w;
        }
      };
      auto element = [&](int e) {
        const int t = e >> 4, rb = t >> 1, tt = t & 1, kb = (e >> 3) & 1, i = e & 7, v = 8 * tt + i;
        const float ds = (float)pf[rb][kb][tt][i] * dp[rb][kb][v];
        if (i & 1) dsf[rb][kb][tt][i >> 1] = pack_bf16x2(dsv, ds);
        else dsv = ds;
      };
      auto mfma = [&](int j, const bf16x8& a) {
        if (j < 32) {
          const int rb = j >> 4, c = (j >> 1) & 7, kb = j & 1;
          dp[rb][kb] = mfma32(a, vreg[kb][c], c ? dp[rb][kb] : nd[rb]);
        } else {
          const int jj = j - 32, t = jj >> 3, nt = (jj >> 1) & 3, kb = jj & 1;
          mfma32_acc<false>(acc[kb][nt], __builtin_bit_cast(bf16x8, dsf[t >> 1][kb][t & 1]), a);  // dS >= 2 slots ago
        }
      };

      load_nd(0);
      static_for<kOpAhead>([&](auto ic) { opq[decltype(ic)::value] = load_op(decltype(ic)::value); });
      static_for<64>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        constexpr int f = j >> 1;
        if constexpr ((j & 1) == 0 && f + kOpAhead < 32) opq[(f + kOpAhead) % (kOpAhead + 1)] = load_op(f + kOpAhead);
        if constexpr (j == 6) load_nd(1);
        // P fragment (rb, kb, tt) three slots before its first element
        static_for<8>([&](auto fc) {
          constexpr int fr = decltype(fc)::value;
          constexpr int rb = fr >> 2, kb = (fr >> 1) & 1, tt = fr & 1;
          if constexpr (b_slot(16 * (2 * rb + tt) + 8 * kb) - 3 == j) pf[rb][kb][tt] = xr[fr * 64 + lane];
        });
        static_for<64>([&](auto ec) {
          constexpr int e = decltype(ec)::value;
          if constexpr (b_slot(e) == j) element(e);
        });
        mfma(j, opq[f % (kOpAhead + 1)]);
        if constexpr (j == 2) dma_piece(dm, 8);
        if constexpr (j >= 3 && j < 11) dma_piece(dm, j - 3);
        __builtin_amdgcn_sched_barrier(0);
      });
    };

    issue_all(2, 1);  // stage -1: the partner computes P of tile 0
    stage_end();
    for (int s = 0; s < ntiles; ++s) {
      stage(sm.qs[s % kQBufs], sm.gs[s % kGBufs], &sm.x[s & 1][pair][0][0], dma_begin(s + 3, s + 2));
      stage_end();
    }
    mfma_drain();
  }
  __builtin_amdgcn_s_waitcnt(0);  // no direct load outlives the workgroup
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc_settle(acc[kb][nt]);  // the reads below stay after the drain

  // ---- write dV (score side) or dK (gradient side, scaled): accumulator
  // column = dim, rows = keys; an item covering part of its keys' query
  // range writes an fp32 partial sum into its slot instead
  const float mul = scorer ? 1.f : p.scale;
  if (tile.slot >= 0) {
    float* part = p.kv_part + ((int64_t)tile.slot * 2 + (scorer ? 0 : 1)) * (kBwdKeys * kHeadDim);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = 64 * pair + 32 * kb + 8 * (v >> 2) + 4 * half + (v & 3);
          part[key * kHeadDim + 32 * nt + qi] = acc[kb][nt][v] * mul;
        }
    return;
  }
  void* out = scorer ? p.dv_step[tile.step] : p.dk_step[tile.step];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = 64 * pair + 32 * kb + 8 * (v >> 2) + 4 * half + (v & 3);
        if (key < tile.nk) {
          const int64_t idx = (key0 + key) * kv_row_stride + tile.kvh * kHeadDim + 32 * nt + qi;
          store_grad(out, idx, acc[kb][nt][v] * mul, p.grad_f32);
        }
      }
}

// Sum of the fp32 partial dV, dK of a split work item's pieces into the
// outputs (one workgroup per split key range; the pieces' slots are
// consecutive).  Keys past nk hold partial sums of clamped copies and are
// not written.
__global__ __launch_bounds__(256) void bwd_kv_reduce_kernel(BwdParams p) {
  const KvSplit sp = p.splits[blockIdx.x];
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  constexpr int kPerSide = kBwdKeys * kHeadDim;
  for (int i = threadIdx.x * 4; i < 2 * kPerSide; i += blockDim.x * 4) {
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < sp.nslots; ++s) {
      const float4 b = *reinterpret_cast<const float4*>(p.kv_part + (int64_t)(sp.slot0 + s) * 2 * kPerSide + i);
      a.x += b.x;
      a.y += b.y;
      a.z += b.z;
      a.w += b.w;
    }
    const int side = i / kPerSide, key = (i % kPerSide) / kHeadDim, d = i % kHeadDim;
    if (key >= sp.nk) continue;
    void* out = side == 0 ? p.dv_step[sp.step] : p.dk_step[sp.step];
    const int64_t idx = (int64_t)(sp.key0 + key) * kv_row_stride + sp.kvh * kHeadDim + d;
    if (p.grad_f32) *reinterpret_cast<float4*>(static_cast<float*>(out) + idx) = a;
    else *reinterpret_cast<bf16x4*>(static_cast<bf16*>(out) + idx) = pack4(a.x, a.y, a.z, a.w);
  }
}

// ------------------------------------------------------------ dq
// One workgroup (4 wavefronts, one per SIMD) per 256-row query tile, as in
// the forward: wavefront w holds rows 64w.. as two 32-row blocks (rb), with
// Q^T and dO^T of its rows (the B operands) and its dQ^T accumulators in the
// accumulation registers.  Per 64-key tile (key blocks kb of 32 keys):
//   S^T = K Q^T, dP^T = V dO^T   (every K or V fragment feeds both row blocks)
//   dS^T = P^T o (dP^T - Delta), P^T = exp2(S^T scale log2e - LSE log2e)
//   dQ^T += K^T dS^T            (every K^T fragment feeds both row blocks)
// The 96 MFMAs of a tile run in six phases of 16 slots,
//   S kb0 | dQ from keys 32..63 of the previous tile | dP kb0 | S kb1 |
//   dP kb1 | dQ from keys 0..31
// with the dS elements of key block 0 computed in the slots of S kb1 and
// dP kb1 and those of key block 1 at the start of the next tile, so the
// vector work runs under the matrix work without a second set of score
// registers.  K/V tiles rotate through three LDS buffers: the previous
// tile's K is still read in the second phase while the next tile arrives.
// The walk runs one loop body: before the first tile a previous tile with
// scores -inf (zero dS) stands in; after the last tile a tail iteration
// runs only the last tile's key block 1 (no MFMA result is left unread,
// whose registers the compiler could reuse while the MFMA still runs).
// Accumulator layout: dQ^T, lane = one query row, rows = dims
// 32*dt + 8*(v/4) + 4*half + v%4.
namespace {

constexpr int kDqBufs = 3;
// FUSED: a query tile's branch-local keys staged in LDS next to the K/V
// buffers for the branch terms (K rows then V rows, kBrPitch apart); a tile
// with more keys computes them from global memory
constexpr int kDqBrSlots = 120;
constexpr int kDqAhead = 3;  // operand fragments read ahead of their MFMAs (two MFMAs each)

// Element e of a key block (32 per lane): the 8-key chunk tt = e/16 (keys
// 16 tt + 8 kb.. in the lane's accumulator slots 8 tt..), row block
// (e/8)%2, slot i = e%8.  Key block 0 of the current tile in slots
// 54..84 (its dQ MFMAs start at 80 and 88; the last dP MFMA of key block 0
// is in slot 47, and its result is read by a vector instruction only after
// the 12 wait states that the compiler would pad); key block 1 of the
// previous tile in slots 0..21 (its dQ MFMAs start at 16 and 24).
constexpr int dq_slot0(int e) { return 54 + (e * 31) / 32; }
constexpr int dq_slot1(int e) { return e < 16 ? e / 2 : 8 + ((e - 16) * 14) / 16; }

}  // namespace

template <int MODE>
__global__ __launch_bounds__(256, 1) void bwd_dq_kernel(BwdParams p) {
  // [buffer][K, V] plane tiles of 64 keys (see tile_off)
  __shared__ __attribute__((aligned(16))) bf16 kvbuf[kDqBufs][2][kFwdKeys * kHeadDim];
  __shared__ __attribute__((aligned(16))) unsigned char brbuf[MODE == kModeFused ? 2 * kDqBrSlots * kBrPitch : 16];
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

  const FwdTile tile = p.qtiles[blockIdx.x];
  const SeqInfo seq = p.seqs[tile.seq];
  if (MODE == kModeStep && !p.acc_first) {
    // a later ring step whose block this tile cannot see leaves the running
    // sums as they are: nothing to load or write
    const int j = ((p.rank - p.step_first) % p.C + p.C) % p.C;
    if (visible_keys(p.toks[tile.tok_begin + tile.ntok - 1].P, j, p.C, seq.c) == 0) return;
  }
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wavefront-uniform
  const int qi = lane & 31;
  const int half = lane >> 5;
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  const LaneOffsets lo = lane_offsets(lane);

  // ---- the lane's two rows (row block rb: row 64 w + 32 rb + qi).  Rows
  // without a token read the rows of the tile's last token (finite data)
  // and take -LSE = -inf, so their probabilities and dS are zero; their dQ
  // is never written.
  int head[2];
  bool valid[2];
  TokInfo tk[2];
  float nl2[2], ndl[2];  // -LSE log2 e, -Delta
  // (the token records and row statistics of both row blocks are read
  // before any Q or dO load is issued: a compiler-visible load after the
  // untracked loads would wait for them too)
  bf16x8 qreg[2][8], greg[2][8];
  const bf16* qp[2];
  const bf16* gp[2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int row = 64 * wave + 32 * rb + qi;
    const int tl = row / p.G;
    head[rb] = tile.kvh * p.G + (row - tl * p.G);
    valid[rb] = tl < tile.ntok;
    const TokInfo tq = p.toks[tile.tok_begin + (valid[rb] ? tl : tile.ntok - 1)];  // one unconditional load
    tk[rb] = valid[rb] ? tq : TokInfo{0, -1, -1, -1};
    const int hq_row = valid[rb] ? head[rb] : tile.kvh * p.G;
    qp[rb] = row_ptr(p.q_main, p.q_br, tq.qrow, p.hq, hq_row);
    gp[rb] = row_ptr(p.do_main, p.do_br, tq.qrow, p.hq, hq_row);
    nl2[rb] = -INFINITY;
    ndl[rb] = 0.f;
    if (valid[rb]) {
      const float2 rs = p.rowstat[(int64_t)(tile.tok_begin + tl) * p.hq + head[rb]];
      nl2[rb] = rs.x;
      ndl[rb] = rs.y;
    }
  }
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      load16_agpr(qreg[rb][c], qp[rb] + 16 * c + 8 * half);
      load16_agpr(greg[rb][c], gp[rb] + 16 * c + 8 * half);
    }
  __builtin_amdgcn_s_waitcnt(0);

  f32x16 dq[2][4];
  if constexpr (MODE == kModeStep) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) mfma32_acc_zero(dq[rb][dt]);
  }

  const int Pmin = p.toks[tile.tok_begin].P;
  const int Pmax = p.toks[tile.tok_begin + tile.ntok - 1].P;

  // ---- FUSED: the dQ accumulators of a branch row start at its
  // branch-local terms, the sum over its branch keys (chain members 0..i,
  // or the whole block; at most BA_MAX_GROUP_LEN, on the vector ALUs) of
  // dS K with P and dS from the row statistics as for a main key.  The
  // scores take the register-held Q and dO (dims 16 c + 8 half + 0..7) and
  // K, V read in that layout; dS K takes K again in the accumulator layout
  // (dims 32 dt + 8 vq + 4 half + 0..3).  The keys come from the tile's
  // staged copy in LDS (the planner's list, each group's keys once); a tile
  // with more than kDqBrSlots keys reads each key's rows from global memory,
  // in one round trip per key.  A lane past its keys (or without any) reads
  // a valid key and gives it weight 0.
  const bool staged = MODE == kModeFused && tile.bk_n > 0 && tile.bk_n <= kDqBrSlots;
  const uint32_t br_lds = lds_addr(&brbuf[0]);
  auto seed_branch = [&](int rb) {
    int nb = 0;
    int bslot = 0;
    GroupInfo gi{0, 1, 0, 0, 0, 0, {0, 0}};
    if (valid[rb] && tk[rb].grp >= 0) {
      gi = p.groups[tk[rb].grp];
      nb = gi.kind == BA_KIND_EAGLE_CHAIN ? tk[rb].gidx + 1 : gi.len;
      if (staged) bslot = p.tok_bslot[tile.tok_begin + (64 * wave + 32 * rb + qi) / p.G];
    }
    f32x16 acc[4];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) acc[dt] = f32x16{};
    if (staged && __ballot(nb > 0)) {
      // the staged keys: LDS reads per key instead of a global round trip
      const uint32_t k0 = br_lds + (uint32_t)bslot * kBrPitch;
      const uint32_t v0 = k0 + (uint32_t)(kDqBrSlots * kBrPitch);
      for (int b = 0; b < BA_MAX_GROUP_LEN; ++b) {
        if (__ballot(b < nb) == 0) break;
        const uint32_t ko = k0 + (uint32_t)min(b, max(nb - 1, 0)) * kBrPitch;
        const uint32_t vo = v0 + (uint32_t)min(b, max(nb - 1, 0)) * kBrPitch;
        float sdot = 0.f, pdot = 0.f;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          sdot = dot8_bf16(qreg[rb][c], lds_ld16(ko + 32u * c + 16u * half), sdot);
          pdot = dot8_bf16(greg[rb][c], lds_ld16(vo + 32u * c + 16u * half), pdot);
        }
        sdot += xor32(sdot);
        pdot += xor32(pdot);
        const float pr = b < nb ? fast_exp2(sdot * p.scale_log2 + nl2[rb]) : 0.f;
        const float ds = pr * (pdot + ndl[rb]);
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int vq = 0; vq < 4; ++vq) {
            const bf16x4 kk = lds_ld8(ko + 64u * dt + 16u * vq + 8u * half);
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[dt][4 * vq + c] += ds * (float)kk[c];
          }
      }
    } else if (__ballot(nb > 0)) {
      for (int b = 0; b < BA_MAX_GROUP_LEN; ++b) {
        if (__ballot(b < nb) == 0) break;
        const int bu = min(b, max(nb - 1, 0));
        int64_t krow = (int64_t)gi.row0 + (int64_t)bu * gi.stride;
        // a row without branch keys (a main row) reads the key of the
        // wavefront's first lane that has one: its weight is zero, and the
        // row it would read otherwise (branch row 0) may belong to no group
        // and hold anything (zero times a non-finite value is not zero)
        {
          const int src = __builtin_ctzll(__ballot(b < nb));  // the loop runs while some lane has a key
          const int lo = __builtin_amdgcn_readlane((int)(krow & 0xffffffff), src);
          const int hi = __builtin_amdgcn_readlane((int)(krow >> 32), src);
          if (nb == 0) krow = (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
        }
        const bf16* kb = p.k_br + krow * kv_row_stride + tile.kvh * kHeadDim;
        const bf16* vb = p.v_br + krow * kv_row_stride + tile.kvh * kHeadDim;
        bf16x8 kd[8], vd[8];
        bf16x4 kk[4][4];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          kd[c] = ld16(kb + 16 * c + 8 * half);
          vd[c] = ld16(vb + 16 * c + 8 * half);
        }
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int vq = 0; vq < 4; ++vq)
            kk[dt][vq] = *reinterpret_cast<const bf16x4*>(kb + 32 * dt + 8 * vq + 4 * half);
        float sdot = 0.f, pdot = 0.f;
#pragma unroll
        for (int c = 0; c < 8; ++c)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            sdot += (float)qreg[rb][c][e] * (float)kd[c][e];
            pdot += (float)greg[rb][c][e] * (float)vd[c][e];
          }
        sdot += xor32(sdot);
        pdot += xor32(pdot);
        const float pr = b < nb ? fast_exp2(sdot * p.scale_log2 + nl2[rb]) : 0.f;
        const float ds = pr * (pdot + ndl[rb]);
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int vq = 0; vq < 4; ++vq)
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[dt][4 * vq + c] += ds * (float)kk[dt][vq][c];
      }
    }
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) asm volatile("" : "=a"(dq[rb][dt]) : "0"(acc[dt]));
  };

  {
    // ---- cursor over (ring step, 64-key tile), as in the forward
    const int step_end = p.step_first + p.step_count;
    auto seek = [&](int i) {
      KvCursor c{i, 0, 0, 0, 0};
      for (; c.i < step_end; ++c.i) {
        c.j = ((p.rank - c.i) % p.C + p.C) % p.C;
        c.lim_hi = visible_keys(Pmax, c.j, p.C, seq.c);
        if (c.lim_hi > 0) break;
      }
      c.lim_lo = visible_keys(Pmin, c.j, p.C, seq.c);
      return c;
    };
    auto next = [&](KvCursor c) {
      if (c.i >= step_end) return c;
      c.kv0 += kFwdKeys;
      return c.kv0 < c.lim_hi ? c : seek(c.i + 1);
    };
    constexpr uint32_t kTileBytes = kFwdKeys * kHeadDim * sizeof(bf16);
    const uint32_t kv_lds = lds_addr(&kvbuf[0][0][0]);
    // direct loads of a tile: 16 per tensor, 4 per wavefront; piece k =
    // 2 m4 + tensor.  The scalar part is computed once per tile, its row
    // bases pinned in scalar registers.
    struct DmaTile {
      const void* kb;
      const void* vb;
      uint32_t dst;
      int nrow;  // rows past the visible prefix repeat its last row
    };
    // the ring block's K/V bases, re-read from the kernel arguments only
    // when the walk moves to another block
    // (their sequence segment and KV head already applied: a tile adds only
    // kv0 rows)
    int cj = -1;
    const bf16* ckb = nullptr;
    const bf16* cvb = nullptr;
    auto dma_tile = [&](const KvCursor& c, int buf) {
      if (c.j != cj) {
        cj = c.j;
        const int64_t seg = (int64_t)seq.seg_off * kv_row_stride + tile.kvh * kHeadDim;
        ckb = p.k_step[cj] + seg;
        cvb = p.v_step[cj] + seg;
        asm volatile("" : "+s"(ckb), "+s"(cvb));
      }
      const int64_t row0 = (int64_t)c.kv0 * kv_row_stride;
      DmaTile d{uniform_ptr(ckb + row0), uniform_ptr(cvb + row0), kv_lds + (uint32_t)(2 * buf) * kTileBytes,
                c.lim_hi - c.kv0};
      asm volatile("" : "+s"(d.kb), "+s"(d.vb));
      return d;
    };
    // a piece's byte offset: row part min(row, nrow - 1) * row stride (the
    // clamp on the row offset itself, the stride being positive) plus the
    // column part, both lane constants precomputed once
    uint32_t frow[4], fcol[4];
#pragma unroll
    for (int m4 = 0; m4 < 4; ++m4) {
      const int m = 4 * wave + m4;
      frow[m4] = (uint32_t)(dma_row<kFwdKeys>(m, lane) * (int)kv_row_stride) * 2u;
      fcol[m4] = (uint32_t)dma_col<kFwdKeys>(m, lane) * 2u;
    }
    auto fetch_piece = [&](const DmaTile& d, int k) {
      const int m4 = k >> 1, tensor = k & 1;
      const int m = 4 * wave + m4;
      const uint32_t lim = (uint32_t)((d.nrow - 1) * (int)kv_row_stride) * 2u;  // wavefront-uniform
      const uint32_t off = min(frow[m4], lim) + fcol[m4];
      dma16_async(tensor ? d.vb : d.kb, off, d.dst + (uint32_t)tensor * kTileBytes + dma_dst_bytes<kFwdKeys>(m));
    };

    // -Delta of the lane's row, the starting value of the dP^T accumulations
    // (dP^T - Delta comes out of the MFMAs)
    f32x16 ndv[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int v = 0; v < 16; ++v) ndv[rb][v] = ndl[rb];

    f32x16 s0[2], s1[2], p0[2], p1[2];  // S^T and dP^T - Delta of key blocks 0 and 1: [rb]
    u32x4 ds0[2][2], ds1[2][2];         // dS^T as bf16 pairs: [rb][tt], B operands of dQ^T
    float sv0 = 0.f, sv1 = 0.f;

    // dS elements of a key block (scores S, dP^T accumulators P, output D)
    auto element = [&](const f32x16 (&S)[2], const f32x16 (&P)[2], u32x4 (&D)[2][2], float& prv, int e) {
      const int tt = e >> 4, rb = (e >> 3) & 1, i = e & 7, v = 8 * tt + i;
      const float pr = fast_exp2(__builtin_fmaf(S[rb][v], p.scale_log2, nl2[rb]));
      const float ds = pr * P[rb][v];
      if (i & 1) {
        uint32_t w = pack_bf16x2(prv, ds);
        asm volatile("" : "+v"(w));  // packed in this slot, not next to the MFMA that reads it
        D[rb][tt][i >> 1] = w;
      } else {
        prv = ds;
      }
    };
    // keys at or past a row's causal limit get score -inf (probability 0)
    auto mask_block = [&](f32x16 (&S)[2], const KvCursor& c, int kb) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const int lim = valid[rb] ? visible_keys(tk[rb].P, c.j, p.C, seq.c) : 0;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int u = c.kv0 + 32 * kb + 8 * (v >> 2) + 4 * half + (v & 3);
          if (u >= lim) S[rb][v] = -INFINITY;
        }
      }
    };

    // One tile iteration.  MFMA j (0..95): phase j/16; fragment j/2 feeds
    // MFMAs j (row block 0) and j+1 (row block 1).  The current tile is in
    // buffer cb, the previous one in pb; mask: apply the causal limits; dn:
    // the tile loaded into the third buffer.
    auto iterate = [&](auto tail_tag, int cb, int pb, const KvCursor& cur, bool mask,
                       const DmaTile& dn) __attribute__((always_inline)) {
      constexpr bool TAIL = decltype(tail_tag)::value;  // phase 1 and key block 1 of the previous tile only
      const bf16* kc = &kvbuf[cb][0][0];
      const bf16* vc = &kvbuf[cb][1][0];
      const bf16* kp = &kvbuf[pb][0][0];
      // K rows and K^T of this tile; V rows and K^T of the previous tile
      const OpBases bk = op_bases(lo, kc, kc);
      const OpBases bv = op_bases(lo, vc, kp);
      auto load_op = [&](int f) -> bf16x8 {
        const int ph = f >> 3, x = f & 7;
        switch (ph) {
          case 0: return row_frag(bk, 0, x);                // K keys 0..31, dims 16x..
          case 1: return tr_frag(bv, 2 + (x >> 2), x & 3);  // K^T of the previous tile, keys 32+16(x/4)..
          case 2: return row_frag(bv, 0, x);                // V keys 0..31
          case 3: return row_frag(bk, 1, x);                // K keys 32..63
          case 4: return row_frag(bv, 1, x);                // V keys 32..63
          default: return tr_frag(bk, x >> 2, x & 3);       // K^T keys 16(x/4)..
        }
      };
      auto mfma = [&](int j, const bf16x8& a) {
        const int ph = j >> 4, jj = j & 15, x = jj >> 1, rb = jj & 1;
        switch (ph) {
          case 0:
            if (x == 0) mfma32_v_first(s0[rb], a, qreg[rb][0]);
            else mfma32_v(s0[rb], a, qreg[rb][x]);
            break;
          // (the tail has no MFMAs before this phase, so its dS packing can
          // sit right before them: padded there)
          case 1: mfma32_acc<TAIL>(dq[rb][x & 3], a, __builtin_bit_cast(bf16x8, ds1[rb][x >> 2])); break;
          case 2:
            if (x == 0) mfma32_v_init<false>(p0[rb], a, greg[rb][0], ndv[rb]);
            else mfma32_v(p0[rb], a, greg[rb][x]);
            break;
          case 3:
            if (x == 0) mfma32_v_first(s1[rb], a, qreg[rb][0]);
            else mfma32_v(s1[rb], a, qreg[rb][x]);
            break;
          case 4:
            if (x == 0) mfma32_v_init<false>(p1[rb], a, greg[rb][0], ndv[rb]);
            else mfma32_v(p1[rb], a, greg[rb][x]);
            break;
          default: mfma32_acc<false>(dq[rb][x & 3], a, __builtin_bit_cast(bf16x8, ds0[rb][x >> 2])); break;
        }
      };
      // fragments f_lo .. f_hi-1 run: all 48, or the 8 of phase 1
      constexpr int f_lo = TAIL ? 8 : 0, f_hi = TAIL ? 16 : 48;
      bf16x8 opq[kDqAhead + 1];  // read-ahead ring
      static_for<kDqAhead>([&](auto fc) {
        constexpr int f = f_lo + decltype(fc)::value;
        opq[f % (kDqAhead + 1)] = load_op(f);
      });
      static_for<96>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        constexpr int f = j >> 1;
        constexpr bool act = f >= f_lo && f < f_hi;
        if constexpr (act && (j & 1) == 0 && f + kDqAhead < f_hi)
          opq[(f + kDqAhead) % (kDqAhead + 1)] = load_op(f + kDqAhead);
        static_for<32>([&](auto ec) {
          constexpr int e = decltype(ec)::value;
          if constexpr (dq_slot1(e) == j) element(s1, p1, ds1, sv1, e);
        });
        if constexpr (!TAIL) {
          if constexpr (j == 24) {
            if (mask) mask_block(s0, cur, 0);
          }
          if constexpr (j == 70) {
            if (mask) mask_block(s1, cur, 1);
          }
          static_for<32>([&](auto ec) {
            constexpr int e = decltype(ec)::value;
            if constexpr (dq_slot0(e) == j) element(s0, p0, ds0, sv0, e);
          });
          // direct loads of tile t+1, in the first slots: its buffer (tile
          // t-2's) is free from the iteration's start
          if constexpr (j < 8) fetch_piece(dn, j);
        }
        if constexpr (act) mfma(j, opq[f % (kDqAhead + 1)]);
        __builtin_amdgcn_sched_barrier(0);
      });
    };

    KvCursor cur = seek(p.step_first);
    if (staged) {
      // the tile's branch keys into LDS (before the first tile's direct
      // loads, which the waits for these loads would otherwise cover too)
      constexpr int kUnroll = 4;
      const int nch = tile.bk_n * 32;  // 16-byte chunks: 16 of K and 16 of V per key
      for (int c0 = tid; c0 < nch; c0 += kUnroll * 256) {
        int32_t krow[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) krow[u] = p.br_keys[tile.bk_off + (min(c0 + u * 256, nch - 1) >> 5)];
        bf16x8 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int part = min(c0 + u * 256, nch - 1) & 31;
          v[u] = ld16((part < 16 ? p.k_br : p.v_br) + (int64_t)krow[u] * kv_row_stride + tile.kvh * kHeadDim +
                      8 * (part & 15));
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int c = c0 + u * 256;
          const int part = c & 31;
          if (c < nch)
            lds_st16(br_lds + (part < 16 ? 0u : (uint32_t)(kDqBrSlots * kBrPitch)) + (uint32_t)(c >> 5) * kBrPitch +
                         16u * (uint32_t)(part & 15),
                     v[u]);
        }
      }
      __syncthreads();
    }
    if (cur.i < step_end) {
      const DmaTile d0 = dma_tile(cur, 0);
#pragma unroll
      for (int k = 0; k < 8; ++k) fetch_piece(d0, k);
    }
    // FUSED: the branch-local terms while the first tile is in flight
    if constexpr (MODE == kModeFused) {
      seed_branch(0);
      seed_branch(1);
    }
    if (cur.i < step_end) {
      // the stand-in previous tile: scores -inf, so its dS are zero
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          s1[rb][v] = -INFINITY;
          p1[rb][v] = 0.f;
        }
      }
      __builtin_amdgcn_s_waitcnt(0);
      lds_barrier();
      int t = 0;
      while (true) {
        const KvCursor nx = next(cur);
        const bool more = nx.i < step_end;
        // with no tile t+1 the loads repeat tile t into the idle buffer
        // (unconditional loads: no branch between the first MFMA slots)
        const DmaTile dn = dma_tile(more ? nx : cur, (t + 1) % kDqBufs);
        const bool mask = cur.kv0 + kFwdKeys > cur.lim_lo;
        // the first tile's stand-in previous tile reads this tile's (finite) K
        iterate(std::false_type{}, t % kDqBufs, t == 0 ? 0 : (t - 1) % kDqBufs, cur, mask, dn);
        wait_vmcnt_lgkm0<0>();  // tile t+1 has landed for this wavefront
        lds_barrier();
        ++t;
        if (!more) break;
        cur = nx;
      }
      // key block 1 of the last tile
      iterate(std::true_type{}, 0, (t - 1) % kDqBufs, cur, false, DmaTile{});
      mfma_drain();  // dQ^T complete before the epilogue reads it
    }
  }
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) acc_settle(dq[rb][dt]);

  // ------------------------------------------------------------ epilogues
  // per row block; every lane runs both so cross-lane exchanges stay uniform
  auto finish = [&](int rb) {
    const int tl = (64 * wave + 32 * rb + qi) / p.G;
    const int64_t acc_row = (int64_t)(tile.tok_begin + tl) * p.hq + head[rb];
    f32x16 st[4];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) st[dt] = dq[rb][dt];
    if (MODE == kModeStep) {
      if (!valid[rb]) return;
      float* dst = p.dq_acc + acc_row * kHeadDim;
      // the running sums of the row, every load issued before any is used
      float4 prev[4][4];
      if (!p.acc_first) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int vq = 0; vq < 4; ++vq)
            prev[dt][vq] = *reinterpret_cast<const float4*>(dst + 32 * dt + 8 * vq + 4 * half);
      } else {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int vq = 0; vq < 4; ++vq) prev[dt][vq] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
          float4 a = prev[dt][vq];
          a.x += st[dt][4 * vq + 0];
          a.y += st[dt][4 * vq + 1];
          a.z += st[dt][4 * vq + 2];
          a.w += st[dt][4 * vq + 3];
          *reinterpret_cast<float4*>(dst + 32 * dt + 8 * vq + 4 * half) = a;
        }
      return;
    }
    if (!valid[rb]) return;

    void* out = tk[rb].qrow >= 0 ? p.dq_main : p.dq_br;
    const int64_t orow = tk[rb].qrow >= 0 ? tk[rb].qrow : -tk[rb].qrow - 1;
    const int64_t base = (orow * p.hq + head[rb]) * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const int64_t o = base + 32 * dt + 8 * vq + 4 * half;
        const float a0 = st[dt][4 * vq] * p.scale, a1 = st[dt][4 * vq + 1] * p.scale;
        const float a2 = st[dt][4 * vq + 2] * p.scale, a3 = st[dt][4 * vq + 3] * p.scale;
        if (p.grad_f32) *reinterpret_cast<float4*>(static_cast<float*>(out) + o) = make_float4(a0, a1, a2, a3);
        else *reinterpret_cast<bf16x4*>(static_cast<bf16*>(out) + o) = pack4(a0, a1, a2, a3);
      }
  };
  finish(0);
  finish(1);
}

// ------------------------------------------------------------ dQ finalize
// Per-step schedule, after the last ring step: dQ of a row is its running
// fp32 sum of dS K over the main keys (the per-step launches), plus for a
// branch row the branch-local terms, times the softmax scale.  One 16-lane
// DPP row per query row (token x head, token order), a lane holding eight
// dims; a branch row recomputes P and dS of its at most 64 branch keys from
// the token-ordered Q and dO copies and the row statistics.
__global__ __launch_bounds__(256) void bwd_dq_finalize_kernel(BwdParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t rows = (int64_t)p.num_tokens * p.hq;
  const int64_t R0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
  const bool live = R0 < rows;
  const int64_t R = live ? R0 : rows - 1;  // rows past the end redo the last row and write nothing
  const int c8 = 8 * (lane & 15);
  const int t = (int)(R / p.hq);
  const int h = (int)(R - (int64_t)t * p.hq);
  const TokInfo tk = p.toks[t];
  const float* da = p.dq_acc + R * kHeadDim + c8;
  const float4 a0 = *reinterpret_cast<const float4*>(da), a1 = *reinterpret_cast<const float4*>(da + 4);
  float acc[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};

  int nb = 0;
  GroupInfo gi{0, 1, 0, 0, 0, 0, {0, 0}};
  if (tk.grp >= 0) {
    gi = p.groups[tk.grp];
    nb = gi.kind == BA_KIND_EAGLE_CHAIN ? tk.gidx + 1 : gi.len;
  }
  if (__ballot(nb > 0) != 0) {  // wavefront-uniform: some row of the wavefront is a branch row
    const bf16x8 qv = ld16(p.qtok + R * kHeadDim + c8), gv = ld16(p.gtok + R * kHeadDim + c8);
    const float2 rs = p.rowstat[R];  // (-LSE log2 e, -Delta)
    float qf[8], gf[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      qf[e] = (float)qv[e];
      gf[e] = (float)gv[e];
    }
    const int64_t kvcol = (int64_t)(h / p.G) * kHeadDim + c8;
    const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
    // keys in groups of four, all four loaded before any is used
    for (int b0 = 0; __ballot(b0 < nb) != 0; b0 += 4) {
      bf16x8 kv[4], vv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        // keys past the row's last read its group's first key (main rows: branch row 0)
        const int64_t krow = (int64_t)gi.row0 + (int64_t)(b0 + u < nb ? b0 + u : 0) * gi.stride;
        kv[u] = ld16(p.k_br + krow * kv_row_stride + kvcol);
        vv[u] = ld16(p.v_br + krow * kv_row_stride + kvcol);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        float sd = 0.f, pd = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          sd = fmaf(qf[e], (float)kv[u][e], sd);
          pd = fmaf(gf[e], (float)vv[u][e], pd);
        }
        sd = row16_sum(sd);
        pd = row16_sum(pd);
        // (after the row sums, which every lane takes part in) a row without
        // this key adds nothing: a main row read branch row 0, which may
        // belong to no group and hold anything
        if (b0 + u >= nb) continue;
        const float pr = fast_exp2(fmaf(sd, p.scale_log2, rs.x));
        const float ds = pr * (pd + rs.y);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf(ds, (float)kv[u][e], acc[e]);
      }
    }
  }
  if (!live) return;
  const int64_t orow = tk.qrow >= 0 ? tk.qrow : -tk.qrow - 1;
  const int64_t o = (orow * p.hq + h) * kHeadDim + c8;
  void* out = tk.qrow >= 0 ? p.dq_main : p.dq_br;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] *= p.scale;
  if (p.grad_f32) {
    float* d = static_cast<float*>(out) + o;
    *reinterpret_cast<float4*>(d) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    *reinterpret_cast<float4*>(d + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
  } else {
    st16(static_cast<bf16*>(out) + o, pack8(acc[0], acc[1], acc[2], acc[3], acc[4], acc[5], acc[6], acc[7]));
  }
}

// ------------------------------------------------------------ branch dK/dV
// One wavefront per (group, KV head, block of four keys).  The wavefront's
// four 16-lane rows each own one key j of the block, a lane holding eight
// dims of K_j, V_j and of the dK_j, dV_j accumulators.  The member x head
// rows (r = i G + h) of the group stream through all four lane rows at once
// from the token-ordered Q and dO copies: every lane row computes its key's
// score and dP with a 16-lane sum, forms P and dS (zero where the key is
// hidden from the member: EAGLE-3 member i sees keys 0..i, a DFlash member
// sees all) and accumulates dS q and P dO.  No atomics and no reduction
// across lanes at the end: lane row j writes dK_j and dV_j once.  Rows are
// loaded four at a time (four heads of one member) before any is used.
namespace {

constexpr int kBrKeys = 4;     // keys per wavefront
constexpr int kBrWaves = 4;
constexpr int kBrRows = 4;     // query rows loaded together

struct BrRow {
  bf16x8 q, g;
  float2 rs;  // (-LSE log2 e, -Delta)
};

}  // namespace

__global__ __launch_bounds__(64 * kBrWaves) void bwd_branch_kernel(BwdParams p, int key_blocks) {
  const int lane = threadIdx.x & 63;
  const int64_t unit = (int64_t)blockIdx.x * kBrWaves + (threadIdx.x >> 6);
  const int64_t gk = unit / key_blocks;
  const int kb = (int)(unit - gk * key_blocks);
  if (gk >= (int64_t)p.num_groups * p.hkv) return;
  const int g = (int)(gk / p.hkv);
  const int kvh = (int)(gk - (int64_t)g * p.hkv);
  const GroupInfo gi = p.groups[g];
  const int n = gi.len;
  if (kb * kBrKeys >= n) return;
  const int G = p.G;
  const bool eagle = gi.kind == BA_KIND_EAGLE_CHAIN;
  const int j = kb * kBrKeys + (lane >> 4);  // this lane row's key
  const int c8 = 8 * (lane & 15);            // this lane's first dim
  const bool has_key = j < n;
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  const int64_t krow = (int64_t)gi.row0 + (int64_t)(has_key ? j : 0) * gi.stride;
  const int64_t kvoff = krow * kv_row_stride + kvh * kHeadDim + c8;
  const bf16x8 kk = ld16(p.k_br + kvoff), vv = ld16(p.v_br + kvoff);
  float kf[8], vf[8], dk[8], dv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    kf[e] = (float)kk[e];
    vf[e] = (float)vv[e];
    dk[e] = 0.f;
    dv[e] = 0.f;
  }
  // members that see at least one key of the block, four heads at a time
  // (a member's G heads are consecutive rows of the token-ordered copies)
  const int i_begin = eagle ? kb * kBrKeys : 0;
  const int64_t head0 = (int64_t)kvh * G;
  for (int i = i_begin; i < n; ++i) {
    const bool vis = has_key && (!eagle || j <= i);
    const int64_t trow0 = (int64_t)(gi.tok0 + i) * p.hq + head0;
    for (int h0 = 0; h0 < G; h0 += kBrRows) {
      BrRow rw[kBrRows];
#pragma unroll
      for (int u = 0; u < kBrRows; ++u) {
        const int64_t trow = trow0 + (h0 + u < G ? h0 + u : h0);
        rw[u] = BrRow{ld16(p.qtok + trow * kHeadDim + c8), ld16(p.gtok + trow * kHeadDim + c8), p.rowstat[trow]};
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the loads together, ahead of their uses
#pragma unroll
      for (int u = 0; u < kBrRows; ++u) {
        float qf[8], gf[8], sd = 0.f, pd = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          qf[e] = (float)rw[u].q[e];
          gf[e] = (float)rw[u].g[e];
          sd = fmaf(qf[e], kf[e], sd);
          pd = fmaf(gf[e], vf[e], pd);
        }
        sd = row16_sum(sd);
        pd = row16_sum(pd);
        const float pr = vis && h0 + u < G ? fast_exp2(fmaf(sd, p.scale_log2, rw[u].rs.x)) : 0.f;  // -LSE log2 e
        const float ds = pr * (pd + rw[u].rs.y);                                                   // -Delta
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          dk[e] = fmaf(ds, qf[e], dk[e]);
          dv[e] = fmaf(pr, gf[e], dv[e]);
        }
      }
    }
  }
  if (!has_key) return;
  if (p.grad_f32) {
    float* dkp = static_cast<float*>(p.dk_br) + kvoff;
    float* dvp = static_cast<float*>(p.dv_br) + kvoff;
    *reinterpret_cast<float4*>(dkp) = make_float4(dk[0] * p.scale, dk[1] * p.scale, dk[2] * p.scale, dk[3] * p.scale);
    *reinterpret_cast<float4*>(dkp + 4) = make_float4(dk[4] * p.scale, dk[5] * p.scale, dk[6] * p.scale, dk[7] * p.scale);
    *reinterpret_cast<float4*>(dvp) = make_float4(dv[0], dv[1], dv[2], dv[3]);
    *reinterpret_cast<float4*>(dvp + 4) = make_float4(dv[4], dv[5], dv[6], dv[7]);
  } else {
    st16(static_cast<bf16*>(p.dk_br) + kvoff, pack8(dk[0] * p.scale, dk[1] * p.scale, dk[2] * p.scale, dk[3] * p.scale,
                                                   dk[4] * p.scale, dk[5] * p.scale, dk[6] * p.scale, dk[7] * p.scale));
    st16(static_cast<bf16*>(p.dv_br) + kvoff, pack8(dv[0], dv[1], dv[2], dv[3], dv[4], dv[5], dv[6], dv[7]));
  }
}

__global__ __launch_bounds__(256) void zero_kernel(uint4* __restrict__ p, int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

static unsigned grid_for(int64_t threads) {
  int64_t b = (threads + 255) / 256;
  return (unsigned)(b < 1 ? 1 : b);
}

hipError_t launch_bwd_preprocess(const BwdParams& p, hipStream_t stream) {
  const int64_t threads = (int64_t)p.num_tokens * p.hq * 16;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(bwd_preprocess_kernel, dim3(grid_for(threads)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_kv(const BwdParams& p, hipStream_t stream) {
  if (p.num_tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(bwd_kv_kernel, dim3(p.num_tiles), dim3(kKvThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_dq(const BwdParams& p, int mode, hipStream_t stream) {
  if (p.num_qtiles == 0) return hipSuccess;
  dim3 grid(p.num_qtiles), block(256);
  if (mode == kModeStep) hipLaunchKernelGGL(bwd_dq_kernel<kModeStep>, grid, block, 0, stream, p);
  else hipLaunchKernelGGL(bwd_dq_kernel<kModeFused>, grid, block, 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_kv_reduce(const BwdParams& p, hipStream_t stream) {
  if (p.num_splits == 0) return hipSuccess;
  hipLaunchKernelGGL(bwd_kv_reduce_kernel, dim3(p.num_splits), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_dq_finalize(const BwdParams& p, hipStream_t stream) {
  const int64_t threads = (int64_t)p.num_tokens * p.hq * 16;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(bwd_dq_finalize_kernel, dim3(grid_for(threads)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_branch(const BwdParams& p, int max_group_len, hipStream_t stream) {
  if (p.num_groups == 0 || max_group_len <= 0) return hipSuccess;
  const int key_blocks = (max_group_len + kBrKeys - 1) / kBrKeys;
  const int64_t units = (int64_t)p.num_groups * p.hkv * key_blocks;
  const int64_t blocks = (units + kBrWaves - 1) / kBrWaves;
  hipLaunchKernelGGL(bwd_branch_kernel, dim3((unsigned)blocks), dim3(64 * kBrWaves), 0, stream, p, key_blocks);
  return hipGetLastError();
}

hipError_t launch_zero(void* ptr, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  const int64_t n16 = (int64_t)(bytes / 16);
  int64_t blocks = (n16 + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, static_cast<uint4*>(ptr), n16);
  return hipGetLastError();
}

}  // namespace ba
