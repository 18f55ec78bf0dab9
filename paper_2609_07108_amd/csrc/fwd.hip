// Forward branch attention for one context-parallel rank share (Sec. 3.2).
//
// One workgroup (4 wavefronts, one per SIMD) owns a query tile of 256 rows:
// up to 256/G query tokens times the G query heads that share one KV head.
// Wavefront w holds rows 64w..64w+63 as two 32-row blocks, so every K and V
// fragment it reads from LDS feeds two MFMAs (one per row block).  Per ring
// step j the tile walks the visible prefix of rank j's KV block in 64-key
// tiles:
//   S^T = K Q^T       (bf16 MFMA 32x32x16, lane = one query row, so the row
//                      maximum is an in-register reduction plus one exchange
//                      with the other half-wavefront)
//   online softmax    (exp2 domain, fp32 statistics)
//   O^T += V^T P^T    (P^T taken straight from the S^T accumulator registers;
//                      V^T read column-wise from the row-major V tile with
//                      transposing LDS reads, in the matching key order)
// The tiles are software-pipelined: while the softmax of tile t runs on the
// vector ALUs, the MFMAs compute S^T of tile t+1 and then O^T += V^T P^T of
// tile t.  K/V tiles arrive by direct global-to-LDS loads into five
// buffers (tiles t+2 and t+3 in flight, one barrier per two tiles).  O^T
// and Q^T live in the accumulation
// registers.  The running maximum used for the exponentials is only moved
// (and O and the row sum rescaled) when a row's maximum grows by more than
// kRescaleSlack in log2 units, so probabilities stay below 2^kRescaleSlack;
// O / l is unchanged by the choice of that reference, so the result is the
// same up to rounding.  Tiles that are fully visible to every row skip the
// mask; the causal limit of a row in block j is a prefix of the block
// because positions increase with the local index (chunk j, then chunk
// 2C-1-j).
//
// Epilogues
//   STEP  : merge the step's partial (O, LSE) into the running fp32 pair in
//           the workspace with Eq. lse-merge (first step writes it); after
//           the last step fwd_finalize_kernel takes the running pair as the
//           main-sequence partial.
//   FUSED : all ring steps in one pass; the running pair stays in registers.
// FUSED and the finalize kernel compute the branch-local partial of every
// branch row (chain members 0..i, or the whole block; at most 64 keys, on
// the vector ALUs), merge it with the main partial by Eq. lse-merge and
// write bf16 O and the natural-log LSE.  In FUSED the tile's branch keys
// (each group's once, listed by the planner) are first copied into the LDS
// that the walk has freed, so a row's keys cost LDS reads rather than a
// chain of dependent global loads per key; the rows then take them eight at
// a time (packed bf16 dot products for the scores, one online-softmax step
// per batch).
#include <type_traits>

#include "ba_internal.h"
#include "device_common.h"
#include "kernels.h"

namespace ba {

namespace {

constexpr float kRescaleSlack = 8.f;  // log2 of the largest probability before a rescale
constexpr int kFragAhead = 2;         // LDS operand fragments read ahead of their MFMAs
constexpr int kKvBufs = 5;  // tiles t-1 .. t+3 (see the walk)
constexpr int kFwdRowBlocks = 1;  // 32-row blocks per wavefront (fwd_kernel's RB)

}  // namespace

// RB: 32-row blocks per wavefront.  RB = 2: four wavefronts (one per SIMD)
// of 64 rows, every K/V fragment read feeding two MFMAs; RB = 1: eight
// wavefronts (two per SIMD) of 32 rows, so that one wavefront's softmax runs
// while the other's MFMAs do (a single wavefront leaves the matrix unit idle
// between its MFMAs), at twice the LDS operand traffic per MFMA.
template <int MODE, int RB>
__global__ __launch_bounds__(512 / RB, 1) void fwd_kernel(FwdParams p) {
  // [buffer][K, V] plane tiles of 64 keys (see tile_off)
  __shared__ __attribute__((aligned(16))) bf16 kvbuf[kKvBufs][2][kFwdKeys * kHeadDim];

  const FwdTile tile = p.tiles[blockIdx.x];
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

  // ---- the lane's two rows (row block rb: row 64 w + 32 rb + qi)
  int head[RB];
  bool valid[RB];
  TokInfo tk[RB];
  // B operand of S^T = K Q^T (Q^T: k = head dims, n = rows), resident in the
  // accumulation registers; rows without a token load a row of the tile's
  // last token (finite, and their results are never written)
  // (the token records of both row blocks are read before any Q load is
  // issued: a compiler-visible load after the untracked Q loads would wait
  // for them too)
  bf16x8 qreg[RB][8];
  const bf16* qptr[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = 32 * RB * wave + 32 * rb + qi;
    const int tl = row / p.G;
    head[rb] = tile.kvh * p.G + (row - tl * p.G);
    valid[rb] = tl < tile.ntok;
    const TokInfo tq = p.toks[tile.tok_begin + (valid[rb] ? tl : tile.ntok - 1)];  // one unconditional load
    tk[rb] = valid[rb] ? tq : TokInfo{0, -1, -1, -1};
    const int hq_row = valid[rb] ? head[rb] : tile.kvh * p.G;
    qptr[rb] = tq.qrow >= 0 ? p.q_main + ((int64_t)tq.qrow * p.hq + hq_row) * kHeadDim
                            : p.q_br + ((int64_t)(-tq.qrow - 1) * p.hq + hq_row) * kHeadDim;
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int c = 0; c < 8; ++c) load16_agpr(qreg[rb][c], qptr[rb] + 16 * c + 8 * half);
  __builtin_amdgcn_s_waitcnt(0);

  f32x16 o[RB][4];  // O^T accumulators, d = 32 dt + 8 (v/4) + 4 half + v%4
  float m_use[RB];  // reference maximum of the exponentials (log2)
  float lsum[RB];   // this lane's share of the row sum
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m_use[rb] = -INFINITY;
    lsum[rb] = 0.f;
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) mfma32_acc_zero(o[rb][dt]);

  const int Pmin = p.toks[tile.tok_begin].P;
  const int Pmax = p.toks[tile.tok_begin + tile.ntok - 1].P;

  {
    // ---- cursor over (ring step, 64-key tile): ring step i brings block
    // j = (rank - i) mod C; tiles cover the prefix of the block that the
    // tile's largest causal limit can see
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
    // direct loads of tile c into buffer buf: 16 per tensor, 4 per
    // wavefront; piece k = 2 m4 + tensor of this wavefront's eight.  The
    // scalar part is computed once per tile and the K and V row bases are
    // pinned in scalar registers: re-reading the ring block's pointer from
    // the kernel arguments per piece would wait on the scalar load, and
    // that wait also drains the LDS operand reads in flight.
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
    for (int m4 = 0; m4 < 2 * RB; ++m4) {
      const int m = 2 * RB * wave + m4;
      frow[m4] = (uint32_t)(dma_row<kFwdKeys>(m, lane) * (int)kv_row_stride) * 2u;
      fcol[m4] = (uint32_t)dma_col<kFwdKeys>(m, lane) * 2u;
    }
    auto fetch_piece = [&](const DmaTile& d, int k) {
      const int m4 = k >> 1, tensor = k & 1;
      const int m = 2 * RB * wave + m4;
      const uint32_t lim = (uint32_t)((d.nrow - 1) * (int)kv_row_stride) * 2u;  // wavefront-uniform
      const uint32_t off = min(frow[m4], lim) + fcol[m4];
      dma16_async(tensor ? d.vb : d.kb, off, d.dst + (uint32_t)tensor * kTileBytes + dma_dst_bytes<kFwdKeys>(m));
    };
    auto fetch = [&](const KvCursor& c, int buf) {
      const DmaTile d = dma_tile(c, buf);
#pragma unroll
      for (int k = 0; k < 4 * RB; ++k) fetch_piece(d, k);
    };

    // ---- LDS fragment reads at a per-tile base address plus a lane
    // constant plus a compile-time offset.  In the plane-tile layout
    // (tile_off) the byte offset of K row 32 kb + qi, dims 16 c + 8 half is
    //   4096 (c / 2) + 2048 kb + 64 qi + 16 ((2 (c % 2) + half) ^ (qi / 4 % 4)),
    // so the lane part takes one of two values (c even / odd); a transposed
    // V read (ld_tr8 with rows 16 t4 + 4 half + i/4 and 16 t4 + 8 + 4 half +
    // i/4, columns 32 dt + (l & 16) + 4 (i % 4), i = l % 16) is at
    //   4096 dt + 1024 t4 + (lane part, one for each of the two row groups).
    const uint32_t q2 = (uint32_t)((qi >> 2) & 3);
    const uint32_t kl0 = 64u * qi + ((((uint32_t)half) ^ q2) << 4);
    const uint32_t kl1 = 64u * qi + ((((uint32_t)half ^ 2u) ^ q2) << 4);
    const uint32_t vl_lo = 2u * (uint32_t)tile_off<kFwdKeys>(4 * half + ((lane & 15) >> 2), (lane & 16) + 4 * (lane & 3));
    const uint32_t vl_hi = 2u * (uint32_t)tile_off<kFwdKeys>(8 + 4 * half + ((lane & 15) >> 2), (lane & 16) + 4 * (lane & 3));
    // The per-tile bases (tile address + lane part) are formed once per tile
    // and hidden from the compiler, which would otherwise fold each read's
    // constant into the tile address first and add the lane part per read.
    struct KBase {
      uint32_t b0, b1;
    };
    struct VBase {
      uint32_t lo, hi;
    };
    auto k_base = [&](uint32_t ks) {
      KBase k{ks + kl0, ks + kl1};
      asm volatile("" : "+v"(k.b0), "+v"(k.b1));
      return k;
    };
    auto v_base = [&](uint32_t vs) {
      VBase v{vs + vl_lo, vs + vl_hi};
      asm volatile("" : "+v"(v.lo), "+v"(v.hi));
      return v;
    };
    // ---- S^T of a tile: fragment f = 8 kb + c (keys 32 kb.., dims 16 c..)
    // feeds both row blocks
    auto s_frag = [&](const KBase& k, int f) -> bf16x8 {
      const int kb = f >> 3, c = f & 7;
      return lds_ld16(((c & 1) ? k.b1 : k.b0) + 4096u * (uint32_t)(c >> 1) + 2048u * (uint32_t)kb);
    };
    auto s_mfma = [&](f32x16 (&S)[RB][2], int f, int rb, const bf16x8& a) {
      const int kb = f >> 3, c = f & 7;
      if (c == 0) mfma32_v_first(S[rb][kb], a, qreg[rb][c]);
      else mfma32_v(S[rb][kb], a, qreg[rb][c]);
    };
    // ---- O^T += V^T P^T: fragment g = 4 t4 + dt (keys 16 t4.., dims 32 dt..);
    // a lane of half h holds keys 16 t4 + 4h + {0..3} and 16 t4 + 8 + 4h +
    // {0..3} in its S^T registers and reads V^T from exactly those rows
    auto v_frag = [&](const VBase& v, int g) -> bf16x8 {
      const int t4 = g >> 2, dt = g & 3;
      const uint32_t o = 4096u * (uint32_t)dt + 1024u * (uint32_t)t4;
      const bf16x4 lo = lds_ld_tr4(v.lo + o), hi = lds_ld_tr4(v.hi + o);
      return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    };

    // maximum of S^T (raw scores) over this lane's 32 keys of a tile (the
    // other 32 keys of the row are in lane l ^ 32); the two halves are only
    // combined when the row's reference maximum may have to move
    auto tile_max = [&](const f32x16 (&S)[RB][2], float (&mx)[RB]) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        float a = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) a = fmaxf(a, S[rb][kb][v]);
        mx[rb] = a;
      }
    };

    // ---- one pipelined iteration on tile t (scores Sc, V in buffer bc):
    // S^T of tile t+1 (K in buffer bn) into Sn, softmax of tile t, then
    // O^T += V^T P^T of tile t; the maximum of tile t+1 is taken at the end.
    // MFMA j in slot j: j < 32 -> S^T fragment j/2, row block j%2;
    // j >= 32 -> V^T fragment (j-32)/2, row block j%2.  Softmax element e
    // (t4 = e/16, row block (e/8)%2, accumulator slot 8 (t4%2) + e%8 of key
    // block t4/2) in slot 52e/64, ahead of the MFMAs of key block t4.
    auto iterate = [&](f32x16 (&Sc)[RB][2], f32x16 (&Sn)[RB][2], uint32_t ks_n, uint32_t vs_c,
                       const float (&m_eff)[RB], float (&mx_n)[RB], auto&& issue_piece) {
      bf16x8 fq[kFragAhead + 1];
      typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
      // packed P^T as bf16 pairs, converted in the element's own slot:
      // [row block][t4] -> the B operand of the t4-th O^T MFMA
      u32x4 pk[RB][4];
      float pv[RB][4][8];
      const KBase kbn = k_base(ks_n);
      const VBase vbc = v_base(vs_c);
      auto frag = [&](int f) -> bf16x8 { return f < 16 ? s_frag(kbn, f) : v_frag(vbc, f - 16); };
      auto element = [&](int e) {
        const int t4 = e / (8 * RB), rb = (e >> 3) % RB, i = e & 7;
        const float x = Sc[rb][t4 >> 1][8 * (t4 & 1) + i];
        const float pr = fast_exp2(__builtin_fmaf(x, p.scale_log2, -m_eff[rb]));
        pv[rb][t4][i] = pr;
        lsum[rb] += pr;  // fp32 probabilities: the LSE bar is tighter than bf16 rounding
        if (i & 1) pk[rb][t4][i >> 1] = pack_bf16x2(pv[rb][t4][i - 1], pr);
      };
      auto pa = [&](int rb, int t4) {
        return __builtin_bit_cast(bf16x8, pk[rb][t4]);
      };
      static_for<kFragAhead>([&](auto fc) { fq[fc.value] = frag(fc.value); });
      static_for<32 * RB>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        constexpr int f = j / RB, rb = j % RB;
        if constexpr (rb == 0 && f + kFragAhead < 32) fq[(f + kFragAhead) % (kFragAhead + 1)] = frag(f + kFragAhead);
        static_for<32 * RB>([&](auto ec) {
          constexpr int e = decltype(ec)::value;
          if constexpr ((e * 26) / 32 == j) element(e);
        });
        if constexpr (j < 16 * RB) {
          s_mfma(Sn, f, rb, fq[f % (kFragAhead + 1)]);
        } else {
          constexpr int g = f - 16, t4 = g >> 2, dt = g & 3;
          mfma32_acc<false>(o[rb][dt], fq[f % (kFragAhead + 1)], pa(rb, t4));  // P^T packed >= 5 slots ago
        }
        if constexpr (j == 32 * RB - 1) tile_max(Sn, mx_n);
        // direct loads of tile t+2, in the first slots: its buffer (tile t-1's)
        // is free from the iteration's start
        if constexpr (j < 4 * RB) issue_piece(j);
        __builtin_amdgcn_sched_barrier(0);
      });
    };

    // ---- apply the causal mask to the scores of a tile that needs it
    auto mask_tile = [&](f32x16 (&S)[RB][2], const KvCursor& c, float (&mx)[RB]) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int lim = valid[rb] ? visible_keys(tk[rb].P, c.j, p.C, seq.c) : 0;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int u = c.kv0 + 32 * kb + 8 * (v >> 2) + 4 * half + (v & 3);
            if (u >= lim) S[rb][kb][v] = -INFINITY;
          }
      }
      tile_max(S, mx);
    };
    // ---- new reference maxima; rescale O and the sums of rows whose
    // maximum moved past the slack (rare after the first tiles)
    // (mx holds half-row maxima: a row moves iff either half asks to, and
    // both halves of the row then take the same, exchanged, maximum)
    auto update_max = [&](const float (&mx)[RB], float (&m_eff)[RB]) {
      float m_new[RB];
      bool move[RB];
      bool any = false;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        m_new[rb] = mx[rb] * p.scale_log2;  // the scale is positive
        any = any || m_new[rb] > m_use[rb] + kRescaleSlack || (m_use[rb] == -INFINITY && m_new[rb] > -INFINITY);
      }
      if (__ballot(any)) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          m_new[rb] = fmaxf(mx[rb], xor32(mx[rb])) * p.scale_log2;
          move[rb] = m_new[rb] > m_use[rb] + kRescaleSlack || (m_use[rb] == -INFINITY && m_new[rb] > -INFINITY);
        }
        mfma_drain();  // pending O^T updates complete before the vector ALUs touch O
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const float alpha = move[rb] ? fast_exp2(m_use[rb] - m_new[rb]) : 1.f;  // m_use = -inf gives 0
          if (move[rb]) m_use[rb] = m_new[rb];
          lsum[rb] *= alpha;
#pragma unroll
          for (int dt = 0; dt < 4; ++dt) acc_scale(o[rb][dt], alpha);
        }
        mfma_drain();
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) m_eff[rb] = m_use[rb] == -INFINITY ? 0.f : m_use[rb];
    };

    KvCursor cur = seek(p.step_first);
    if (cur.i < step_end) {
      KvCursor nxt = next(cur);
      KvCursor nx2 = next(nxt);
      fetch(cur, 0);
      if (nxt.i < step_end) fetch(nxt, 1);
      if (nx2.i < step_end) fetch(nx2, 2);
      __builtin_amdgcn_s_waitcnt(0);
      lds_barrier();
      f32x16 Sa[RB][2], Sb[RB][2];
      float mx[RB], m_eff[RB];
      // prologue: S^T of the first tile
      static_for<16 * RB>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        s_mfma(Sa, j / RB, j % RB, s_frag(k_base(kv_lds), j / RB));
      });
      mfma_drain();  // the scores are read by the vector ALUs next
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) vacc_settle(Sa[rb][kb]);
      tile_max(Sa, mx);
      int t = 0;
      // Tile t is in buffer t % 5; scores of tile t in Sa (t even) or Sb.
      // Iteration t reads K of tile t+1 and V of tile t and loads tile t+3
      // into the buffer of tile t-2, which no wavefront reads after the
      // last barrier; only odd iterations wait for their loads and
      // synchronise, which publishes tiles t+2 and t+3 for the next pair.
      auto step = [&](f32x16 (&Sc)[RB][2], f32x16 (&Sn)[RB][2], auto sync) {
        const KvCursor n3 = next(nx2);
        // with no tile t+3 the loads repeat tile t into the idle buffer
        const KvCursor ld = n3.i < step_end ? n3 : cur;
        const DmaTile d3 = dma_tile(ld, (t + 3) % kKvBufs);
        if (cur.kv0 + kFwdKeys > cur.lim_lo) mask_tile(Sc, cur, mx);
        update_max(mx, m_eff);
        // with no tile t+1 the S^T MFMAs read a stale buffer and are discarded
        iterate(Sc, Sn, kv_lds + (uint32_t)((t + 1) % kKvBufs) * 2u * kTileBytes,
                kv_lds + (uint32_t)(t % kKvBufs) * 2u * kTileBytes + kTileBytes, m_eff, mx,
                [&](int k) { fetch_piece(d3, k); });
        if constexpr (decltype(sync)::value) {
          wait_vmcnt_lgkm0<0>();  // tiles t+2 and t+3 have landed for this wavefront
          lds_barrier();
        }
        cur = nxt;
        nxt = nx2;
        nx2 = n3;
        ++t;
      };
      while (true) {
        step(Sa, Sb, std::false_type{});
        if (cur.i >= step_end) break;
        step(Sb, Sa, std::true_type{});
        if (cur.i >= step_end) break;
      }
      wait_vmcnt_lgkm0<0>();  // no direct load outlives the walk (after an even iteration some are in flight)
      mfma_drain();  // O^T complete before the epilogue reads it
    }
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) acc_settle(o[rb][dt]);

  // ------------------------------------------------------------ epilogues
  // per row block; every lane runs all of them so cross-lane exchanges stay uniform
  float l_tot[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) l_tot[rb] = lsum[rb] + xor32(lsum[rb]);

  // FUSED: the branch-local keys of the tile's tokens (each group's once,
  // listed by the planner) staged in the LDS that the key walk has freed, K
  // rows then V rows; a tile with more than kBrSlots of them (bk_n < 0)
  // reads them from global memory per row instead
  const bool staged = MODE == kModeFused && tile.bk_n > 0;
  const uint32_t br_lds = lds_addr(&kvbuf[0][0][0]);
  if (staged) {
    constexpr int kThreads = 512 / RB;
    constexpr int kUnroll = 4;
    __syncthreads();  // every wavefront is past its last read of the K/V buffers
    const int nch = tile.bk_n * 32;  // 16-byte chunks: 16 of K and 16 of V per key
    // the thread index recomputed (no register holds it across the walk)
    const int t_id = 64 * wave + (int)__lane_id();
    for (int c0 = t_id; c0 < nch; c0 += kUnroll * kThreads) {
      int32_t krow[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) krow[u] = p.br_keys[tile.bk_off + (min(c0 + u * kThreads, nch - 1) >> 5)];
      bf16x8 v[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int part = min(c0 + u * kThreads, nch - 1) & 31;
        v[u] = ld16((part < 16 ? p.k_br : p.v_br) + (int64_t)krow[u] * kv_row_stride + tile.kvh * kHeadDim +
                    8 * (part & 15));
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = c0 + u * kThreads;
        const int part = c & 31;
        if (c < nch)
          lds_st16(br_lds + (part < 16 ? 0u : (uint32_t)(kBrSlots * kBrPitch)) + (uint32_t)(c >> 5) * kBrPitch +
                       16u * (uint32_t)(part & 15),
                   v[u]);
      }
    }
    __syncthreads();
  }

  auto finish = [&](int rb) {
    const int64_t acc_row = (int64_t)(tile.tok_begin + (32 * RB * wave + 32 * rb + qi) / p.G) * p.hq + head[rb];

    if (MODE == kModeStep) {
      if (!valid[rb]) return;
      f32x16 st_o[4];
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) st_o[dt] = o[rb][dt];
      float* oacc = p.o_acc + acc_row * kHeadDim;
      if (l_tot[rb] > 0.f) {
        const float lse2 = m_use[rb] + __log2f(l_tot[rb]);
        const float inv = 1.f / l_tot[rb];
        float wa = 0.f, wb = inv;
        float lse_new = lse2;
        // the running pair of the row, every load issued before any is used
        float4 prev[4][4];
        float la = -INFINITY;
        if (!p.acc_first) {
#pragma unroll
          for (int dt = 0; dt < 4; ++dt)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq)
              prev[dt][vq] = *reinterpret_cast<const float4*>(oacc + 32 * dt + 8 * vq + 4 * half);
          la = p.lse_acc[acc_row];
          const float hi = fmaxf(la, lse2);
          const float ea = fast_exp2(la - hi);  // la = -inf gives 0
          const float eb = fast_exp2(lse2 - hi);
          const float tot = ea + eb;
          lse_new = hi + __log2f(tot);
          wa = ea / tot;
          wb = eb / tot * inv;
        } else {
#pragma unroll
          for (int dt = 0; dt < 4; ++dt)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq) prev[dt][vq] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
          for (int vq = 0; vq < 4; ++vq) {
            const float4 pr = prev[dt][vq];
            float4 r;
            r.x = wa * pr.x + wb * st_o[dt][4 * vq + 0];
            r.y = wa * pr.y + wb * st_o[dt][4 * vq + 1];
            r.z = wa * pr.z + wb * st_o[dt][4 * vq + 2];
            r.w = wa * pr.w + wb * st_o[dt][4 * vq + 3];
            *reinterpret_cast<float4*>(oacc + 32 * dt + 8 * vq + 4 * half) = r;
          }
        }
        if (half == 0) p.lse_acc[acc_row] = lse_new;
      } else if (p.acc_first) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int vq = 0; vq < 4; ++vq)
            *reinterpret_cast<float4*>(oacc + 32 * dt + 8 * vq + 4 * half) = make_float4(0.f, 0.f, 0.f, 0.f);
        if (half == 0) p.lse_acc[acc_row] = -INFINITY;
      }
      return;
    }

    // main-sequence partial: LSE (log2) in lse_m; O^T stays in the
    // accumulation registers until the output is written, normalised by
    // inv there
    float lse_m, inv = 0.f;
    if (l_tot[rb] > 0.f) {
      lse_m = m_use[rb] + __log2f(l_tot[rb]);
      inv = 1.f / l_tot[rb];
    } else {
      lse_m = -INFINITY;
    }

    // ---- branch-local partial (vector ALUs; at most 64 keys per row)
    int nb = 0;
    int bslot = 0;
    GroupInfo gi{0, 1, 0, 0, 0, 0, {0, 0}};
    if (valid[rb] && tk[rb].grp >= 0) {
      gi = p.groups[tk[rb].grp];
      nb = gi.kind == BA_KIND_EAGLE_CHAIN ? tk[rb].gidx + 1 : gi.len;
      if (staged) bslot = p.tok_bslot[tile.tok_begin + (32 * RB * wave + 32 * rb + qi) / p.G];
    }
    float mb = -INFINITY, lb = 0.f;
    f32x16 ob[4];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) ob[dt] = f32x16{};
    if (staged) {
      // keys in batches of eight from the staged rows: the row's Q read once,
      // one online-softmax step per batch; a lane past its keys reads a
      // valid slot and gives it probability 0
      constexpr int kBatch = 8;
      const uint32_t kb0 = br_lds + (uint32_t)bslot * kBrPitch + 16u * (uint32_t)half;
      const uint32_t vb0 = br_lds + (uint32_t)(kBrSlots * kBrPitch) + (uint32_t)bslot * kBrPitch + 8u * (uint32_t)half;
      for (int b0 = 0; b0 < BA_MAX_GROUP_LEN; b0 += kBatch) {
        if (__ballot(b0 < nb) == 0) break;
        int key[kBatch];
#pragma unroll
        for (int k = 0; k < kBatch; ++k) key[k] = min(b0 + k, max(nb - 1, 0));
        float dot[kBatch];
#pragma unroll
        for (int k = 0; k < kBatch; ++k) dot[k] = 0.f;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const bf16x8 qv = ld16(qptr[rb] + 16 * c + 8 * half);  // L2-resident
#pragma unroll
          for (int k = 0; k < kBatch; ++k) {
            const bf16x8 kv = lds_ld16(kb0 + (uint32_t)key[k] * kBrPitch + 32u * (uint32_t)c);
            dot[k] = dot8_bf16(qv, kv, dot[k]);
          }
        }
        float x[kBatch];
        float m_new = mb;
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
          dot[k] += xor32(dot[k]);
          x[k] = b0 + k < nb ? dot[k] * p.scale_log2 : -INFINITY;
          m_new = fmaxf(m_new, x[k]);
        }
        if (m_new == -INFINITY) continue;  // no key of this lane's row in the batch
        const float alpha = fast_exp2(mb - m_new);  // mb = -inf gives 0
        mb = m_new;
        lb *= alpha;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) ob[dt] *= alpha;
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
          const float e = fast_exp2(x[k] - m_new);  // x = -inf gives 0
          lb += e;
#pragma unroll
          for (int dt = 0; dt < 4; ++dt)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq) {
              const bf16x4 vv = lds_ld8(vb0 + (uint32_t)key[k] * kBrPitch + 64u * (uint32_t)dt + 16u * (uint32_t)vq);
#pragma unroll
              for (int c = 0; c < 4; ++c) ob[dt][4 * vq + c] += e * (float)vv[c];
            }
        }
      }
    }
    for (int b = 0; b < (staged ? 0 : BA_MAX_GROUP_LEN); ++b) {
      const bool active = b < nb;
      if (__ballot(active) == 0) break;
      const int64_t krow = (int64_t)gi.row0 + (int64_t)b * gi.stride;
      const bf16* kb = p.k_br + krow * kv_row_stride + tile.kvh * kHeadDim;
      const bf16* vb = p.v_br + krow * kv_row_stride + tile.kvh * kHeadDim;
      float dot = 0.f;
      if (active) {
        // the row's Q is re-read (L2-resident) rather than kept in the
        // accumulation registers past the key walk, which would make the
        // compiler spill them around it
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const bf16x8 kv = ld16(kb + 16 * c + 8 * half);
          const bf16x8 qv = ld16(qptr[rb] + 16 * c + 8 * half);
#pragma unroll
          for (int e = 0; e < 8; ++e) dot += (float)qv[e] * (float)kv[e];
        }
      }
      dot += xor32(dot);
      if (!active) continue;
      const float x = dot * p.scale_log2;
      const float m_new = fmaxf(mb, x);
      const float alpha = fast_exp2(mb - m_new);
      const float e = fast_exp2(x - m_new);
      lb = lb * alpha + e;
      mb = m_new;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
          const bf16x4 vv = *reinterpret_cast<const bf16x4*>(vb + 32 * dt + 8 * vq + 4 * half);
#pragma unroll
          for (int c = 0; c < 4; ++c) ob[dt][4 * vq + c] = ob[dt][4 * vq + c] * alpha + e * (float)vv[c];
        }
      }
    }
    if (!valid[rb]) return;

    // ---- Eq. lse-merge of the main and branch partials, then write out
    const float lse_b = lb > 0.f ? mb + __log2f(lb) : -INFINITY;
    const float hi = fmaxf(lse_m, lse_b);
    const float wm = lse_m == -INFINITY ? 0.f : fast_exp2(lse_m - hi);
    const float wbr = lse_b == -INFINITY ? 0.f : fast_exp2(lse_b - hi);
    const float tot = wm + wbr;
    const float lse2 = hi + __log2f(tot);
    const float cm = wm / tot * inv;
    const float cb = lb > 0.f ? wbr / (tot * lb) : 0.f;

    bf16* out;
    float* lse_out;
    if (tk[rb].qrow >= 0) {
      out = p.o_main + ((int64_t)tk[rb].qrow * p.hq + head[rb]) * kHeadDim;
      lse_out = p.lse_main + (int64_t)head[rb] * p.n_local + tk[rb].qrow;
    } else {
      const int64_t br = -tk[rb].qrow - 1;
      out = p.o_br + (br * p.hq + head[rb]) * kHeadDim;
      lse_out = p.lse_br + (int64_t)head[rb] * p.n_br + br;
    }
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const int v = 4 * vq;
        *reinterpret_cast<bf16x4*>(out + 32 * dt + 8 * vq + 4 * half) =
            pack4(cm * o[rb][dt][v] + cb * ob[dt][v], cm * o[rb][dt][v + 1] + cb * ob[dt][v + 1],
                  cm * o[rb][dt][v + 2] + cb * ob[dt][v + 2], cm * o[rb][dt][v + 3] + cb * ob[dt][v + 3]);
      }
    if (half == 0) *lse_out = lse2 * kLn2;
  };
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) finish(rb);
}

// ------------------------------------------------------------ finalize
// Per-step schedule, after the last ring step: the running pair (O, LSE) of
// every query row is its main-sequence partial.  One 16-lane DPP row per
// query row (token x head, token order), a lane holding eight dims.  Branch
// rows add their branch-local partial (online softmax over chain members
// 0..i or the whole block, at most 64 keys) and merge it with the main
// partial by Eq. lse-merge; every row is written as bf16 O and natural-log
// LSE.  Memory-bound: the running fp32 O is read once, O written once.
__global__ __launch_bounds__(256) void fwd_finalize_kernel(FwdParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t rows = (int64_t)p.num_tokens * p.hq;
  const int64_t R0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
  const bool live = R0 < rows;
  const int64_t R = live ? R0 : rows - 1;  // rows past the end redo the last row and write nothing
  const int c8 = 8 * (lane & 15);
  const int t = (int)(R / p.hq);
  const int h = (int)(R - (int64_t)t * p.hq);
  const TokInfo tk = p.toks[t];
  const float* oa = p.o_acc + R * kHeadDim + c8;
  const float4 a0 = *reinterpret_cast<const float4*>(oa), a1 = *reinterpret_cast<const float4*>(oa + 4);
  const float om[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
  const float lse_m = p.lse_acc[R];  // log2 units; -inf: no main key

  int nb = 0;
  GroupInfo gi{0, 1, 0, 0, 0, 0, {0, 0}};
  if (tk.grp >= 0) {
    gi = p.groups[tk.grp];
    nb = gi.kind == BA_KIND_EAGLE_CHAIN ? tk.gidx + 1 : gi.len;
  }
  float mb = -INFINITY, lb = 0.f, ob[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) ob[e] = 0.f;
  if (__ballot(nb > 0) != 0) {  // wavefront-uniform: some row of the wavefront is a branch row
    const int64_t qr = tk.qrow >= 0 ? tk.qrow : -tk.qrow - 1;
    const bf16x8 qv = ld16((tk.qrow >= 0 ? p.q_main : p.q_br) + (qr * p.hq + h) * kHeadDim + c8);
    float qf[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) qf[e] = (float)qv[e];
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
      float x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) dot = fmaf(qf[e], (float)kv[u][e], dot);
        dot = row16_sum(dot);  // every lane takes part in the row sum
        x[u] = b0 + u < nb ? dot * p.scale_log2 : -INFINITY;
      }
      if (b0 < nb) {
        const float m_new = fmaxf(fmaxf(mb, fmaxf(x[0], x[1])), fmaxf(x[2], x[3]));
        const float alpha = fast_exp2(mb - m_new);  // mb = -inf at the first key: 0
        float ex[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) ex[u] = fast_exp2(x[u] - m_new);  // keys past the last: 0
        lb = lb * alpha + ((ex[0] + ex[1]) + (ex[2] + ex[3]));
        mb = m_new;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          ob[e] = fmaf(ob[e], alpha,
                       fmaf(ex[0], (float)vv[0][e],
                            fmaf(ex[1], (float)vv[1][e], fmaf(ex[2], (float)vv[2][e], ex[3] * (float)vv[3][e]))));
      }
    }
  }
  if (!live) return;

  // Eq. lse-merge of the main and branch partials (log2 units)
  const float lse_b = lb > 0.f ? mb + __log2f(lb) : -INFINITY;
  const float hi = fmaxf(lse_m, lse_b);
  const float wm = lse_m == -INFINITY ? 0.f : fast_exp2(lse_m - hi);
  const float wbr = lse_b == -INFINITY ? 0.f : fast_exp2(lse_b - hi);
  const float tot = wm + wbr;
  const float lse2 = tot > 0.f ? hi + __log2f(tot) : -INFINITY;
  const float cm = tot > 0.f ? wm / tot : 0.f;
  const float cb = lb > 0.f ? wbr / (tot * lb) : 0.f;
  bf16* out;
  float* lse_out;
  if (tk.qrow >= 0) {
    out = p.o_main + ((int64_t)tk.qrow * p.hq + h) * kHeadDim;
    lse_out = p.lse_main + (int64_t)h * p.n_local + tk.qrow;
  } else {
    const int64_t br = -tk.qrow - 1;
    out = p.o_br + (br * p.hq + h) * kHeadDim;
    lse_out = p.lse_br + (int64_t)h * p.n_br + br;
  }
  st16(out + c8, pack8(cm * om[0] + cb * ob[0], cm * om[1] + cb * ob[1], cm * om[2] + cb * ob[2],
                       cm * om[3] + cb * ob[3], cm * om[4] + cb * ob[4], cm * om[5] + cb * ob[5],
                       cm * om[6] + cb * ob[6], cm * om[7] + cb * ob[7]));
  if ((lane & 15) == 0) *lse_out = lse2 * kLn2;
}

hipError_t launch_fwd_finalize(const FwdParams& p, hipStream_t stream) {
  const int64_t threads = (int64_t)p.num_tokens * p.hq * 16;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(fwd_finalize_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_fwd(const FwdParams& p, int mode, hipStream_t stream) {
  if (p.num_tiles == 0) return hipSuccess;
  dim3 grid(p.num_tiles), block(256);
  block = dim3(512 / kFwdRowBlocks);
  if (mode == kModeStep) hipLaunchKernelGGL((fwd_kernel<kModeStep, kFwdRowBlocks>), grid, block, 0, stream, p);
  else hipLaunchKernelGGL((fwd_kernel<kModeFused, kFwdRowBlocks>), grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace ba
