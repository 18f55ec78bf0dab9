// Backward branch attention for one context-parallel rank share (Sec. 3.2:
// the backward pass replays the same KV ring and accumulates gradients
// locally).
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
//   dq         : dQ, query-tile parallel like the forward: per key tile
//                S^T = K Q^T, dP^T = V dO^T, dS^T, dQ^T += K^T dS^T, with the
//                branch-local keys handled in the epilogue.  Splitting dQ off
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

}  // namespace

// ------------------------------------------------------------ preprocess
// 32 lanes per (token, head): -Delta = -<dO, O> over 128 dims and -LSE in
// log2 units (both stored negated so the dK/dV kernel can start its S and dP
// accumulations from them); Q and dO rows are also copied into token order, so the
// dK/dV kernel addresses a query tile without indirection.
__global__ __launch_bounds__(256) void bwd_preprocess_kernel(BwdParams p) {
  const int64_t pair = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 5;
  const int sub = threadIdx.x & 31;
  if (pair >= (int64_t)p.num_tokens * p.hq) return;
  const int32_t t = (int32_t)(pair / p.hq);
  const int32_t head = (int32_t)(pair - (int64_t)t * p.hq);
  const TokInfo tk = p.toks[t];
  const bf16* o = row_ptr(p.o_main, p.o_br, tk.qrow, p.hq, head);
  const bf16* g = row_ptr(p.do_main, p.do_br, tk.qrow, p.hq, head);
  const bf16x4 ov = reinterpret_cast<const bf16x4*>(o)[sub];
  const bf16x4 gv = reinterpret_cast<const bf16x4*>(g)[sub];
  const bf16x4 qv = reinterpret_cast<const bf16x4*>(row_ptr(p.q_main, p.q_br, tk.qrow, p.hq, head))[sub];
  reinterpret_cast<bf16x4*>(p.qtok + pair * kHeadDim)[sub] = qv;
  reinterpret_cast<bf16x4*>(p.gtok + pair * kHeadDim)[sub] = gv;
  float dlt = (float)ov[0] * (float)gv[0] + (float)ov[1] * (float)gv[1] + (float)ov[2] * (float)gv[2] +
              (float)ov[3] * (float)gv[3];
#pragma unroll
  for (int m = 16; m >= 1; m >>= 1) dlt += __shfl_xor(dlt, m, 32);
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
//   score wavefront (w = p):     K scale log2e of the pair's keys in
//                                registers; S' = Q (K scale log2e)^T - LSE
//                                log2e (the accumulation starts from -LSE
//                                log2e), P = exp2(S') with the causal mask,
//                                P handed to the partner through LDS,
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
// are walked in order.  In stage i the score wavefronts compute P of tile
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
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
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
  // also loads the tile's LSE, 1 its causal limits, 2 its -Delta.  Rows
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
  // Q of tile kq (score wavefronts) or dO of tile kg (gradient wavefronts);
  // past the last tile the last one again, into the tile's own (idle)
  // buffer.  A stage's loads go out in 9 pieces spread over its schedule:
  // pieces 0-7 are the row loads (rows 32 pair + 16 (piece/4) + lane/4,
  // plane piece%4), piece 8 the statistic.
  const bf16* rows_src = scorer ? p.qtok : p.gtok;
  asm volatile("" : "+s"(rows_src));  // kept in registers, not re-read per stage
  struct DmaStage {
    int qt0, nt;
    uint32_t b;
  };
  auto dma_begin = [&](int kq, int kg) __attribute__((always_inline)) {
    const int k = scorer ? kq : kg;
    DmaStage d;
    d.qt0 = tile.q_begin + (k < ntiles ? k : ntiles - 1) * tpt;
    d.nt = tile.q_end - d.qt0;  // tokens left from qt0
    d.b = scorer ? q_lds + (uint32_t)(k % kQBufs) * (uint32_t)sizeof(QSide)
                 : g_lds + (uint32_t)(k % kGBufs) * (uint32_t)sizeof(GSide);
    return d;
  };
  auto dma_piece = [&](const DmaStage& d, int piece) __attribute__((always_inline)) {
    if (piece == 8) {
      const bool ok = stl < tpt && stl < d.nt;
      if (wave == 1) {
        const void* base = uniform_ptr(p.toks + d.qt0);
        const uint32_t off = (uint32_t)((ok ? stl : p.num_tokens - d.qt0) * (int)sizeof(TokInfo) +
                                        (int)offsetof(TokInfo, P));
        dma4_async(base, off, d.b + (uint32_t)offsetof(QSide, pl));
      } else if (wave != 3) {
        const void* base = uniform_ptr(p.rowstat + (int64_t)d.qt0 * p.hq + head0);
        const uint32_t off = (uint32_t)((ok ? stl * p.hq + shg : 0) * (int)sizeof(float2) + (wave == 0 ? 0 : 4));
        dma4_async(base, off, d.b + (uint32_t)(wave == 0 ? offsetof(QSide, l2) : offsetof(GSide, nd)));
      }
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
  // loads of this stage (9 for wavefronts 0-2, 8 for wavefront 3) stay in
  // flight.  The barrier publishes everything to the workgroup.
  auto stage_end = [&]() __attribute__((always_inline)) {
    if (wave == 3) wait_vmcnt_lgkm0<8>();
    else wait_vmcnt_lgkm0<9>();
    lds_barrier();
  };

  // Operand fragments of a 64-row plane tile sit at compile-time offsets
  // from four per-lane bases: row fragments (rows 32 rb + qi, columns
  // 16 c + 8h; the chunk permutation depends on c only through its parity)
  // from row_even / row_odd, transposed fragments (rows 16 t + 4h + {0..3}
  // and 16 t + 8 + 4h + {0..3}, columns 32 nt + ..) from tr_lo / tr_hi.
  const int row_even = tile_off<kBwdRows>(qi, 8 * half);
  const int row_odd = tile_off<kBwdRows>(qi, 16 + 8 * half);
  const int trc = (lane & 16) + 4 * (lane & 3);
  const int tr_lo = tile_off<kBwdRows>(4 * half + ((lane & 15) >> 2), trc);
  const int tr_hi = tile_off<kBwdRows>(8 + 4 * half + ((lane & 15) >> 2), trc);
  // A stage's four bases (LDS byte addresses) are opaque to the compiler, so
  // it cannot re-associate the constant offsets into per-fragment registers.
  struct OpBases {
    uint32_t re, ro, tl, th;
  };
  auto op_bases = [&](const bf16* rowT, const bf16* trT) __attribute__((always_inline)) {
    OpBases o{lds_lane_addr(rowT + row_even), lds_lane_addr(rowT + row_odd), lds_lane_addr(trT + tr_lo),
              lds_lane_addr(trT + tr_hi)};
    asm volatile("" : "+v"(o.re), "+v"(o.ro), "+v"(o.tl), "+v"(o.th));
    return o;
  };
  auto row_frag = [&](const OpBases& o, int rb, int c) __attribute__((always_inline)) {
    return lds_ld16(((c & 1) ? o.ro : o.re) + (uint32_t)(((c >> 1) * kBwdRows + 32 * rb) * 64));
  };
  auto tr_frag = [&](const OpBases& o, int t, int nt) __attribute__((always_inline)) {
    const uint32_t off = (uint32_t)((nt * kBwdRows + 16 * t) * 64);
    const bf16x4 lo = lds_ld_tr4(o.tl + off), hi = lds_ld_tr4(o.th + off);
    return bf16x8(__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };

  // Tiles [t_lo, t_hi) need no mask: every row has a token and sees all
  // keys of the block (tokens from q_full on do).
  int t_lo = ntiles, t_hi = ntiles;
  if (tile.nk == kBwdKeys && tpt * G == kBwdRows) {
    t_lo = min(ntiles, max(0, (tile.q_full - tile.q_begin + tpt - 1) / tpt));
    t_hi = max(t_lo, (tile.q_end - tile.q_begin) / tpt);
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
    // K scale log2e of the lane's keys (B operands of S'), resident in the
    // accumulation registers.  Rounding the scaled K to bf16 perturbs each
    // score by about 2^-9 of |q| |k| scale (relative), well inside the
    // gradients' tolerance, and saves one multiply-add per probability.
    bf16x8 kreg[2][8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const bf16x8 kr = ld16(kvsrc + (key0 + kload[kb]) * kv_row_stride + 16 * c + 8 * half);
        bf16x8 ks;
#pragma unroll
        for (int e = 0; e < 8; ++e) ks[e] = (bf16)((float)kr[e] * p.scale_log2);
        asm volatile("" : "=a"(kreg[kb][c]) : "0"(ks));
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

      const OpBases ob = op_bases(qn.q, gc.g);
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
        float pr = fast_exp2(s[rb][kb][v]);
        if (MASK) {
          const int lim = c == 0 ? sp[rb][q].x : c == 1 ? sp[rb][q].y : c == 2 ? sp[rb][q].z : sp[rb][q].w;
          pr = kpos[kb] <= lim ? pr : 0.f;
        }
        if (v & 1) pn[rb][kb][v >> 3][(v & 7) >> 1] = __builtin_bit_cast(uint32_t, bf16x2{(bf16)prv, (bf16)pr});
        else prv = pr;
      };
      auto mfma = [&](int j, const bf16x8& a) {
        if (j < 32) {
          const int rb = j >> 4, c = (j >> 1) & 7, kb = j & 1;
          if (c == 0) mfma32_v_init(s[rb][kb], a, kreg[kb][0], nl[rb]);
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
        if constexpr ((j & 7) == 4) dma_piece(dm, j >> 3);
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

      const OpBases ob = op_bases(gc.g, qc.q);
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
        if (i & 1) dsf[rb][kb][tt][i >> 1] = __builtin_bit_cast(uint32_t, bf16x2{(bf16)dsv, (bf16)ds});
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
        if constexpr ((j & 7) == 4) dma_piece(dm, j >> 3);
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
  // column = dim, rows = keys
  void* out = scorer ? p.dv_step[tile.step] : p.dk_step[tile.step];
  const float mul = scorer ? 1.f : p.scale;
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

// ------------------------------------------------------------ dq
// Half a forward query tile, 128 rows (4 wavefronts x 32), per workgroup.
// Accumulator layout: dQ^T, lane = one query row, rows = dims
// 32*dt + 8*(v/4) + 4*half + v%4.
template <int MODE>
__global__ __launch_bounds__(256, 2) void bwd_dq_kernel(BwdParams p) {
  // [buffer][K, V] plane tiles of 64 keys (see tile_off), double-buffered
  __shared__ __attribute__((aligned(16))) bf16 kvbuf[2][2][kFwdKeys * kHeadDim];

  // two workgroups per query tile, rows [128 h, 128 h + 128) of it.  Block
  // 16 g + 8 h + x takes half h of tile 8 g + x: workgroups go to the 8 XCDs
  // round-robin by index, so both halves of a tile run on one XCD and share
  // its L2 for the K/V tiles they both stream
  const int qt = 8 * (blockIdx.x >> 4) + (blockIdx.x & 7);
  if (qt >= p.num_qtiles) return;
  const FwdTile tile = p.qtiles[qt];
  const int rbase = 128 * ((blockIdx.x >> 3) & 1);
  if (rbase / p.G >= tile.ntok) return;  // no token in this half
  const SeqInfo seq = p.seqs[tile.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wavefront-uniform
  const int qi = lane & 31;
  const int half = lane >> 5;
  const int row = rbase + wave * 32 + qi;
  const int tl = row / p.G;
  const int head = tile.kvh * p.G + (row - tl * p.G);
  const bool valid = tl < tile.ntok;
  TokInfo tk;
  if (valid) tk = p.toks[tile.tok_begin + tl];
  else tk = TokInfo{0, -1, -1, -1};
  const int64_t acc_row = (int64_t)(tile.tok_begin + tl) * p.hq + head;

  bf16x8 qreg[8], greg[8];
  float nl2 = 0.f, ndl = 0.f;  // -LSE log2 e, -Delta
  if (valid) {
    const bf16* qp = row_ptr(p.q_main, p.q_br, tk.qrow, p.hq, head);
    const bf16* gp = row_ptr(p.do_main, p.do_br, tk.qrow, p.hq, head);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      qreg[c] = ld16(qp + 16 * c + 8 * half);
      greg[c] = ld16(gp + 16 * c + 8 * half);
    }
    const float2 rs = p.rowstat[acc_row];
    nl2 = rs.x;
    ndl = rs.y;
  } else {
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      qreg[c] = bf16x8{};
      greg[c] = bf16x8{};
    }
  }

  f32x16 dq[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) dq[dt] = f32x16{};

  const int Pmin = p.toks[tile.tok_begin + rbase / p.G].P;
  const int Pmax = p.toks[tile.tok_begin + min(tile.ntok - 1, (rbase + 127) / p.G)].P;
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;

  if (MODE != kModeFinal) {
    // One 64-key tile: S^T = K Q^T, dP^T = V dO^T, dS^T, dQ^T += K^T dS^T.
    // MASK (compile time) only on tiles crossing some row's causal limit.
    auto compute = [&](int j, int kv0, const bf16* ks, const bf16* vs, auto mask_tag) {
      constexpr bool MASK = decltype(mask_tag)::value;
      const int my_lim = valid ? visible_keys(tk.P, j, p.C, seq.c) : 0;
      f32x16 s[2], dp[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        s[kt] = f32x16{};
        dp[kt] = f32x16{};
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          s[kt] = mfma32(ld16(&ks[tile_off<kFwdKeys>(32 * kt + qi, 16 * c + 8 * half)]), qreg[c], s[kt]);
          dp[kt] = mfma32(ld16(&vs[tile_off<kFwdKeys>(32 * kt + qi, 16 * c + 8 * half)]), greg[c], dp[kt]);
        }
      }
      // ---- dS^T = P^T (dP^T - Delta), P^T = exp2(S^T scale log2e - LSE log2e)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float pr = fast_exp2(__builtin_fmaf(s[kt][v], p.scale_log2, nl2));
          if (MASK) {
            const int u = kv0 + 32 * kt + 8 * (v >> 2) + 4 * half + (v & 3);
            pr = u < my_lim ? pr : 0.f;
          }
          dp[kt][v] = pr * (dp[kt][v] + ndl);
        }
      // ---- dQ^T += K^T dS^T: k-block t = keys 16t.. of the tile; the lane's
      // dS^T values of half h are keys 16t+4h+{0..3}, 16t+8+4h+{0..3}
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const f32x16& src = dp[t >> 1];
        const int v0 = 8 * (t & 1);
        const bf16x8 b = pack8(src[v0], src[v0 + 1], src[v0 + 2], src[v0 + 3], src[v0 + 4], src[v0 + 5],
                               src[v0 + 6], src[v0 + 7]);
        const int ka = 16 * t + 4 * half, kb = ka + 8;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) dq[dt] = mfma32(ld_tr8<kFwdKeys>(ks, 32 * dt, ka, kb, lane), b, dq[dt]);
      }
    };
    walk_kv_tiles(p, seq, tile.kvh, Pmax, wave, lane, kvbuf, [&](int j, int kv0, const bf16* ks, const bf16* vs) {
      if (kv0 + kFwdKeys <= visible_keys(Pmin, j, p.C, seq.c)) compute(j, kv0, ks, vs, std::false_type{});
      else compute(j, kv0, ks, vs, std::true_type{});
    });
  }

  if (MODE == kModeStep) {
    if (!valid) return;
    float* dst = p.dq_acc + acc_row * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        float4* d4 = reinterpret_cast<float4*>(dst + 32 * dt + 8 * vq + 4 * half);
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
        if (!p.acc_first) a = *d4;
        a.x += dq[dt][4 * vq + 0];
        a.y += dq[dt][4 * vq + 1];
        a.z += dq[dt][4 * vq + 2];
        a.w += dq[dt][4 * vq + 3];
        *d4 = a;
      }
    return;
  }
  if (MODE == kModeFinal && valid) {
    const float* src = p.dq_acc + acc_row * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const float4 a = *reinterpret_cast<const float4*>(src + 32 * dt + 8 * vq + 4 * half);
        dq[dt][4 * vq + 0] = a.x;
        dq[dt][4 * vq + 1] = a.y;
        dq[dt][4 * vq + 2] = a.z;
        dq[dt][4 * vq + 3] = a.w;
      }
  }

  // ---- branch-local keys of this row (vector ALUs)
  int nb = 0;
  GroupInfo gi{0, 1, 0, 0, 0, {0, 0, 0}};
  if (valid && tk.grp >= 0) {
    gi = p.groups[tk.grp];
    nb = gi.kind == BA_KIND_EAGLE_CHAIN ? tk.gidx + 1 : gi.len;
  }
  for (int b = 0; b < BA_MAX_GROUP_LEN; ++b) {
    const bool active = b < nb;
    if (__ballot(active) == 0) break;
    const int64_t krow = (int64_t)gi.row0 + (int64_t)b * gi.stride;
    const bf16* kb = p.k_br + krow * kv_row_stride + tile.kvh * kHeadDim;
    const bf16* vb = p.v_br + krow * kv_row_stride + tile.kvh * kHeadDim;
    float sdot = 0.f, pdot = 0.f;
    if (active) {
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const bf16x8 kv = ld16(kb + 16 * c + 8 * half);
        const bf16x8 vv = ld16(vb + 16 * c + 8 * half);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          sdot += (float)qreg[c][e] * (float)kv[e];
          pdot += (float)greg[c][e] * (float)vv[e];
        }
      }
    }
    sdot += xor32(sdot);
    pdot += xor32(pdot);
    if (!active) continue;
    const float pr = fast_exp2(sdot * p.scale_log2 + nl2);
    const float ds = pr * (pdot + ndl);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const bf16x4 kk = *reinterpret_cast<const bf16x4*>(kb + 32 * dt + 8 * vq + 4 * half);
#pragma unroll
        for (int c = 0; c < 4; ++c) dq[dt][4 * vq + c] += ds * (float)kk[c];
      }
  }
  if (!valid) return;

  void* out = tk.qrow >= 0 ? p.dq_main : p.dq_br;
  const int64_t orow = tk.qrow >= 0 ? tk.qrow : -tk.qrow - 1;
  const int64_t base = (orow * p.hq + head) * kHeadDim;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int vq = 0; vq < 4; ++vq) {
      const int64_t o = base + 32 * dt + 8 * vq + 4 * half;
      const float a0 = dq[dt][4 * vq] * p.scale, a1 = dq[dt][4 * vq + 1] * p.scale;
      const float a2 = dq[dt][4 * vq + 2] * p.scale, a3 = dq[dt][4 * vq + 3] * p.scale;
      if (p.grad_f32) *reinterpret_cast<float4*>(static_cast<float*>(out) + o) = make_float4(a0, a1, a2, a3);
      else *reinterpret_cast<bf16x4*>(static_cast<bf16*>(out) + o) = pack4(a0, a1, a2, a3);
    }
}

// ------------------------------------------------------------ branch dK/dV
// One workgroup per (group, KV head).  Each wavefront takes query rows
// (member i, head) in turn; lanes hold two dims each and every score needs a
// wavefront-wide reduction.  The group's dK/dV are summed in LDS (fp32) and
// written once.
__global__ __launch_bounds__(256) void bwd_branch_kernel(BwdParams p) {
  extern __shared__ float acc_s[];  // [2][len][128]: dK sums, dV sums
  const int g = blockIdx.x / p.hkv;
  const int kvh = blockIdx.x - g * p.hkv;
  const GroupInfo gi = p.groups[g];
  const int n = gi.len;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < 2 * n * kHeadDim; i += blockDim.x) acc_s[i] = 0.f;
  __syncthreads();
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  const int G = p.G;
  for (int rr = wave; rr < n * G; rr += 4) {
    const int i = rr / G;
    const int head = kvh * G + (rr - i * G);
    const int64_t brow = (int64_t)gi.row0 + (int64_t)i * gi.stride;
    const bf16* q = p.q_br + (brow * p.hq + head) * kHeadDim;
    const bf16* g_ = p.do_br + (brow * p.hq + head) * kHeadDim;
    const float2 rs = p.rowstat[(int64_t)(gi.tok0 + i) * p.hq + head];
    const float q0 = (float)q[2 * lane], q1 = (float)q[2 * lane + 1];
    const float g0 = (float)g_[2 * lane], g1 = (float)g_[2 * lane + 1];
    const int nk = gi.kind == BA_KIND_EAGLE_CHAIN ? i + 1 : n;
    for (int j = 0; j < nk; ++j) {
      const int64_t krow = (int64_t)gi.row0 + (int64_t)j * gi.stride;
      const bf16* kp = p.k_br + krow * kv_row_stride + kvh * kHeadDim;
      const bf16* vp = p.v_br + krow * kv_row_stride + kvh * kHeadDim;
      float sdot = q0 * (float)kp[2 * lane] + q1 * (float)kp[2 * lane + 1];
      float pdot = g0 * (float)vp[2 * lane] + g1 * (float)vp[2 * lane + 1];
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        sdot += __shfl_xor(sdot, m);
        pdot += __shfl_xor(pdot, m);
      }
      const float pr = fast_exp2(sdot * p.scale_log2 + rs.x);  // rs.x = -LSE log2 e
      const float ds = pr * (pdot + rs.y);  // rs.y = -Delta
      atomicAdd(&acc_s[j * kHeadDim + 2 * lane], ds * q0);
      atomicAdd(&acc_s[j * kHeadDim + 2 * lane + 1], ds * q1);
      atomicAdd(&acc_s[(n + j) * kHeadDim + 2 * lane], pr * g0);
      atomicAdd(&acc_s[(n + j) * kHeadDim + 2 * lane + 1], pr * g1);
    }
  }
  __syncthreads();
  for (int idx = tid; idx < n * kHeadDim; idx += blockDim.x) {
    const int j = idx / kHeadDim, d = idx - j * kHeadDim;
    const int64_t krow = (int64_t)gi.row0 + (int64_t)j * gi.stride;
    const int64_t o = krow * kv_row_stride + kvh * kHeadDim + d;
    store_grad(p.dk_br, o, acc_s[idx] * p.scale, p.grad_f32);
    store_grad(p.dv_br, o, acc_s[n * kHeadDim + idx], p.grad_f32);
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
  const int64_t threads = (int64_t)p.num_tokens * p.hq * 32;
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
  dim3 grid(16 * ((p.num_qtiles + 7) / 8)), block(256);  // see the block mapping in the kernel
  if (mode == kModeStep) hipLaunchKernelGGL(bwd_dq_kernel<kModeStep>, grid, block, 0, stream, p);
  else if (mode == kModeFinal) hipLaunchKernelGGL(bwd_dq_kernel<kModeFinal>, grid, block, 0, stream, p);
  else hipLaunchKernelGGL(bwd_dq_kernel<kModeFused>, grid, block, 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_branch(const BwdParams& p, int max_group_len, hipStream_t stream) {
  if (p.num_groups == 0) return hipSuccess;
  const size_t lds = (size_t)2 * max_group_len * kHeadDim * sizeof(float);
  hipLaunchKernelGGL(bwd_branch_kernel, dim3(p.num_groups * p.hkv), dim3(256), lds, stream, p);
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
