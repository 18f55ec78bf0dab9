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
//   preprocess : Delta and LSE * log2(e) per (query token, head).
//   kv         : dK and dV.  One workgroup per 128 keys of one ring-step
//                block, sequence and KV head (dK/dV in registers); it walks
//                the query tokens that reach those keys in 64-row tiles
//                (tokens x the G heads of the KV head), double-buffered in
//                LDS by direct global-to-LDS loads.  No atomics.
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
// 32 lanes per (token, head): Delta = <dO, O> over 128 dims and the row's
// LSE in log2 units; Q and dO rows are also copied into token order, so the
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
    p.rowstat[pair] = make_float2(lse * kLog2e, dlt);
  }
}

// ------------------------------------------------------------ kv (ring)
// Workgroup of 4 wavefronts (one per SIMD, up to 512 registers each) on 128
// keys: wavefront w owns keys 32w..32w+31 against every 64-row query tile
// (tokens x the G heads of the KV head).  K and V of its keys stay in
// registers (B operands of S = Q K^T and dP = dO V^T), dK and dV accumulate
// in registers.  No atomics.
//
// Query tiles (Q and dO plane tiles plus per-row LSE, Delta and causal
// limit) rotate through three LDS buffers: while tile i is processed, tile
// i+1 is resident and tile i+2 in flight.  Every global access of the loop
// is such a direct load, at addresses computed from the token index alone
// (token-ordered copies of Q and dO), so the loop has no compiler-visible
// memory loads and the waits on the loads are explicit.
//
// Inside a stage the 64 MFMAs run in a fixed order -- S/dP of row block 0,
// S/dP of row block 1, dV/dK over the four 16-row reduction blocks -- each
// preceded by the LDS read of the operand kOpAhead MFMAs later and, from
// the 17th on, by one softmax element, so that the exponentials overlap the
// matrix work and no LDS latency is exposed.
namespace {

constexpr int kKvWaves = 4;
constexpr int kKvThreads = 64 * kKvWaves;
constexpr int kOpAhead = 4;
constexpr int kDmaPerStage = 8;  // Q/dO direct loads of one wavefront per tile

struct QTileLds {
  bf16 q[kBwdRows * kHeadDim];
  bf16 g[kBwdRows * kHeadDim];
  float l2[kBwdRows];  // LSE * log2 e
  float dl[kBwdRows];  // Delta
  int pl[kBwdRows];    // causal limit P (-1: no token)
};

}  // namespace

__global__ __launch_bounds__(kKvThreads, 1) void bwd_kv_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) QTileLds qs[3];

  const BwdTile tile = p.tiles[blockIdx.x];
  const SeqInfo seq = p.seqs[tile.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wavefront-uniform
  const int qi = lane & 31;
  const int half = lane >> 5;
  const int G = p.G;
  const int tpt = kBwdRows / G;  // tokens per query tile
  const int ntiles = (tile.q_end - tile.q_begin + tpt - 1) / tpt;  // >= 1 (planner)
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  const int64_t key0 = (int64_t)seq.seg_off + tile.u0;  // first key row in the block
  const int head0 = tile.kvh * G;

  // ---- this lane's key: its position decides visibility (visible to a row
  // iff position <= the row's causal limit; local index < c lies in chunk
  // `step`, the rest in chunk 2C-1-step)
  const int my_key = 32 * wave + qi;
  const int kload = my_key < tile.nk ? my_key : tile.nk - 1;
  int kpos;
  {
    const int u = tile.u0 + my_key;
    kpos = u < seq.c ? tile.step * seq.c + u : (2 * p.C - 1 - tile.step) * seq.c + (u - seq.c);
    if (my_key >= tile.nk) kpos = 0x7fffffff;
  }

  // ---- direct-load rows: lane carries tile rows 32*(w%2) + 16j + lane/4
  // (j = 0, 1) of Q (wavefronts 0-1) or dO (2-3); wavefronts 0-2 also load
  // one statistic of row `lane`.  Rows without a token read the tile's first
  // row (finite data) and the sentinel token's limit -1.
  const bf16* src = wave >= 2 ? p.gtok : p.qtok;
  int dtl[2], dhg[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = 32 * (wave & 1) + 16 * j + (lane >> 2);
    dtl[j] = row / G;
    dhg[j] = row - dtl[j] * G;
  }
  const int stl = lane / G, shg = lane - stl * G;
  const uint32_t qs_lds = lds_addr(&qs[0]);
  auto issue = [&](int t) {
    const uint32_t b = qs_lds + (uint32_t)(t % 3) * (uint32_t)sizeof(QTileLds);
    // past the end: the last tile again, into the idle buffer
    const int qt0 = tile.q_begin + (t < ntiles ? t : ntiles - 1) * tpt;
    const int nt = tile.q_end - qt0;  // tokens left from qt0
    if (wave < 3) {
      const bool ok = stl < tpt && stl < nt;
      if (wave == 2) {
        const void* base = uniform_ptr(p.toks + qt0);
        const uint32_t off = (uint32_t)((ok ? stl : p.num_tokens - qt0) * (int)sizeof(TokInfo) +
                                        (int)offsetof(TokInfo, P));
        dma4_async(base, off, b + (uint32_t)offsetof(QTileLds, pl));
      } else {
        const void* base = uniform_ptr(p.rowstat + (int64_t)qt0 * p.hq + head0);
        const uint32_t off = (uint32_t)((ok ? stl * p.hq + shg : 0) * (int)sizeof(float2) + 4 * wave);
        dma4_async(base, off, b + (uint32_t)(wave == 0 ? offsetof(QTileLds, l2) : offsetof(QTileLds, dl)));
      }
    }
    const uint32_t dst = b + (uint32_t)(wave >= 2 ? offsetof(QTileLds, g) : offsetof(QTileLds, q));
    const void* base = uniform_ptr(src + ((int64_t)qt0 * p.hq + head0) * kHeadDim);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const bool ok = dtl[j] < tpt && dtl[j] < nt;
      const int r = ok ? dtl[j] * p.hq + dhg[j] : 0;  // row relative to (qt0, head0)
#pragma unroll
      for (int pl = 0; pl < 4; ++pl) {
        const int m = 8 * (wave & 1) + 4 * j + pl;
        const uint32_t off = (uint32_t)(r * kHeadDim + dma_col<kBwdRows>(m, lane)) * (uint32_t)sizeof(bf16);
        dma16_async(base, off, dst + dma_dst_bytes<kBwdRows>(m));
      }
    }
  };

  bf16x8 kreg[8], vreg[8];
  {
    const bf16* kp = p.k_step[tile.step] + (key0 + kload) * kv_row_stride + tile.kvh * kHeadDim;
    const bf16* vp = p.v_step[tile.step] + (key0 + kload) * kv_row_stride + tile.kvh * kHeadDim;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      kreg[c] = ld16(kp + 16 * c + 8 * half);
      vreg[c] = ld16(vp + 16 * c + 8 * half);
    }
  }
  f32x16 dk[4], dv[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    mfma32_acc_zero(dk[nt]);
    mfma32_acc_zero(dv[nt]);
  }
  issue(0);
  issue(1);
  __builtin_amdgcn_s_waitcnt(0);
  lds_barrier();

  // ---- the stage.  MFMA j: j < 32 -> S (even j) / dP (odd j) of row block
  // j/16, reduction chunk (j/2)%8; j >= 32 -> dV (even) / dK (odd), column
  // block ((j-32)/2)%4, reduction block t = (j-32)/8 (query rows 16t..16t+15;
  // a lane of half h holds rows 16t+4h+{0..3} and 16t+8+4h+{0..3}, so the
  // dO / Q operand is read column-wise from the same rows).
  // Softmax element e (slot 16+e): accumulator slot e%16 of row block e/16,
  // query row 32(e/16) + 8((e%16)/4) + 4h + e%4.
  auto stage = [&](const QTileLds& cur, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    f32x16 s[2], dp[2];
    bf16x8 opq[kOpAhead + 1];
    float4 sl[8], sd[8];
    int4 sp[8];
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    bf16x2 pp[16], pd[16];
    float prv = 0.f, dsv = 0.f;

    auto load_op = [&](int j) -> bf16x8 {
      if (j < 32) {
        const int off = tile_off<kBwdRows>(32 * (j >> 4) + qi, 16 * ((j >> 1) & 7) + 8 * half);
        return ld16((j & 1) ? &cur.g[off] : &cur.q[off]);
      }
      const int jj = j - 32, t = jj >> 3, nt = (jj >> 1) & 3;
      return ld_tr8<kBwdRows>((jj & 1) ? cur.q : cur.g, 32 * nt, 16 * t + 4 * half, 16 * t + 8 + 4 * half,
                              lane);
    };
    auto load_stats = [&](int q) {
      const int r0 = 32 * (q >> 2) + 8 * (q & 3) + 4 * half;
      sl[q] = *reinterpret_cast<const float4*>(&cur.l2[r0]);
      sd[q] = *reinterpret_cast<const float4*>(&cur.dl[r0]);
      if (MASK) sp[q] = *reinterpret_cast<const int4*>(&cur.pl[r0]);
    };
    auto softmax = [&](int e) {
      const int mt = e >> 4, v = e & 15, q = e >> 2, c = e & 3;
      const float l = c == 0 ? sl[q].x : c == 1 ? sl[q].y : c == 2 ? sl[q].z : sl[q].w;
      const float d = c == 0 ? sd[q].x : c == 1 ? sd[q].y : c == 2 ? sd[q].z : sd[q].w;
      float pr = fast_exp2(__builtin_fmaf(s[mt][v], p.scale_log2, -l));
      if (MASK) {
        const int lim = c == 0 ? sp[q].x : c == 1 ? sp[q].y : c == 2 ? sp[q].z : sp[q].w;
        pr = kpos <= lim ? pr : 0.f;
      }
      const float ds = pr * (dp[mt][v] - d);
      if (e & 1) {
        pp[e >> 1] = bf16x2{(bf16)prv, (bf16)pr};
        pd[e >> 1] = bf16x2{(bf16)dsv, (bf16)ds};
      } else {
        prv = pr;
        dsv = ds;
      }
    };
    auto pa = [&](int t) {
      return bf16x8{pp[4 * t][0], pp[4 * t][1], pp[4 * t + 1][0], pp[4 * t + 1][1],
                    pp[4 * t + 2][0], pp[4 * t + 2][1], pp[4 * t + 3][0], pp[4 * t + 3][1]};
    };
    auto dsa = [&](int t) {
      return bf16x8{pd[4 * t][0], pd[4 * t][1], pd[4 * t + 1][0], pd[4 * t + 1][1],
                    pd[4 * t + 2][0], pd[4 * t + 2][1], pd[4 * t + 3][0], pd[4 * t + 3][1]};
    };
    auto mfma = [&](int j, const bf16x8& a) {
      if (j < 32) {
        const int mt = j >> 4, c = (j >> 1) & 7;
        if (j & 1) dp[mt] = mfma32(a, vreg[c], c ? dp[mt] : f32x16{});
        else s[mt] = mfma32(a, kreg[c], c ? s[mt] : f32x16{});
      } else {
        const int jj = j - 32, t = jj >> 3, nt = (jj >> 1) & 3;
        if (jj & 1) mfma32_acc(dk[nt], dsa(t), a);
        else mfma32_acc(dv[nt], pa(t), a);
      }
    };

    static_for<kOpAhead>([&](auto jc) { opq[jc.value] = load_op(jc.value); });
    static_for<64>([&](auto jc) {
      constexpr int j = decltype(jc)::value;
      if constexpr (j + kOpAhead < 64) opq[(j + kOpAhead) % (kOpAhead + 1)] = load_op(j + kOpAhead);
      if constexpr (j >= 12 && j < 44 && (j & 3) == 0) load_stats((j - 12) >> 2);
      if constexpr (j >= 16 && j < 48) softmax(j - 16);
      mfma(j, opq[j % (kOpAhead + 1)]);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  // Tiles [t_lo, t_hi) need no mask: every row has a token and sees all
  // keys of the block (tokens from q_full on do).  The three ranges run as
  // separate loops so each has one stage variant and the accumulators stay
  // in place across iterations.
  int t_lo = ntiles, t_hi = ntiles;
  if (tile.nk == kBwdKeys && tpt * G == kBwdRows) {
    t_lo = min(ntiles, max(0, (tile.q_full - tile.q_begin + tpt - 1) / tpt));
    t_hi = max(t_lo, (tile.q_end - tile.q_begin) / tpt);
  }
  auto run = [&](int t0, int t1, auto mask_tag) {
    for (int it = t0; it < t1; ++it) {
      issue(it + 2);
      stage(qs[it % 3], mask_tag);
      // tile it+1 (issued one stage ago) has landed for this wavefront; the
      // loads of tile it+2 stay in flight
      wait_vmcnt_lgkm0<kDmaPerStage>();
      lds_barrier();
    }
    mfma_drain();  // accumulators settled before the compiler may move them
  };
  run(0, t_lo, std::true_type{});
  run(t_lo, t_hi, std::false_type{});
  run(t_hi, ntiles, std::true_type{});
  __builtin_amdgcn_s_waitcnt(0);  // no direct load outlives the workgroup
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {  // the reads below stay after the last drain
    acc_settle(dk[nt]);
    acc_settle(dv[nt]);
  }

  // ---- write dK (scaled) and dV: accumulator column = dim, rows = keys
  void* dkout = p.dk_step[tile.step];
  void* dvout = p.dv_step[tile.step];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int key = 32 * wave + 8 * (v >> 2) + 4 * half + (v & 3);
      if (key < tile.nk) {
        const int64_t idx = (key0 + key) * kv_row_stride + tile.kvh * kHeadDim + 32 * nt + qi;
        store_grad(dkout, idx, dk[nt][v] * p.scale, p.grad_f32);
        store_grad(dvout, idx, dv[nt][v], p.grad_f32);
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
  float lse2 = 0.f, dlt = 0.f;
  if (valid) {
    const bf16* qp = row_ptr(p.q_main, p.q_br, tk.qrow, p.hq, head);
    const bf16* gp = row_ptr(p.do_main, p.do_br, tk.qrow, p.hq, head);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      qreg[c] = ld16(qp + 16 * c + 8 * half);
      greg[c] = ld16(gp + 16 * c + 8 * half);
    }
    const float2 rs = p.rowstat[acc_row];
    lse2 = rs.x;
    dlt = rs.y;
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
          float pr = fast_exp2(__builtin_fmaf(s[kt][v], p.scale_log2, -lse2));
          if (MASK) {
            const int u = kv0 + 32 * kt + 8 * (v >> 2) + 4 * half + (v & 3);
            pr = u < my_lim ? pr : 0.f;
          }
          dp[kt][v] = pr * (dp[kt][v] - dlt);
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
    const float pr = fast_exp2(sdot * p.scale_log2 - lse2);
    const float ds = pr * (pdot - dlt);
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
      const float pr = fast_exp2(sdot * p.scale_log2 - rs.x);
      const float ds = pr * (pdot - rs.y);
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
