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
// 32 lanes per (token, head): Delta = <dO, O> over 128 dims, and the row's
// LSE in log2 units.
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
// Workgroup of 4 wavefronts (one per SIMD, so up to 512 registers each) on
// 128 keys: wavefront w owns keys 32w..32w+31 against every 64-row query
// tile.  K and V of its keys stay in registers (B operands of S = Q K^T and
// dP = dO V^T), dK and dV accumulate in registers.  Query tiles (Q and dO)
// are double-buffered plane tiles (see tile_off) fetched with direct
// global-to-LDS loads while the previous one is in use; the loop is unrolled
// by two so that each half works on a fixed buffer.
namespace {

constexpr int kKvWaves = 4;
constexpr int kKvThreads = 64 * kKvWaves;

struct QTileLds {
  bf16 q[kBwdRows * kHeadDim];
  bf16 g[kBwdRows * kHeadDim];
  float l2[kBwdRows];
  float dl[kBwdRows];
  int lim[kBwdRows];
};

struct RowStats {
  float l2, dl;
  int lim;
};

// Issue the direct loads of the query tile starting at token qt0 into `s`:
// wavefronts 0-1 fetch Q, 2-3 dO, eight loads of 16 rows x 32 columns each.
// Rows without a token (past the range, or past tpt*G) fetch the tile's
// first row: their probabilities are masked to zero, so only finiteness
// matters.  Threads 0..63 also return the row statistics, written to LDS
// once the buffer is no longer read.
__device__ __forceinline__ RowStats fetch_qtile(const BwdParams& p, const BwdTile& tile, const SeqInfo& seq,
                                               int qt0, int tid, QTileLds& s) {
  const int G = p.G;
  const int tpt = kBwdRows / G;
  const int lane = tid & 63, wave = tid >> 6;
  const bool is_do = wave >= 2;
  const bf16* mainp = is_do ? p.do_main : p.q_main;
  const bf16* brp = is_do ? p.do_br : p.q_br;
  bf16* dst = is_do ? s.g : s.q;
#pragma unroll
  for (int m8 = 0; m8 < 8; ++m8) {
    const int m = 8 * (wave & 1) + m8;
    const int row = dma_row<kBwdRows>(m, lane);
    const int tl = row / G;
    const int tok = qt0 + tl;
    const bool ok = tl < tpt && tok < tile.q_end;
    const TokInfo tk = p.toks[ok ? tok : qt0];
    const int head = tile.kvh * G + (ok ? row - tl * G : 0);
    dma16(row_ptr(mainp, brp, tk.qrow, p.hq, head) + dma_col<kBwdRows>(m, lane), dma_dst<kBwdRows>(dst, m));
  }
  RowStats r{0.f, 0.f, 0};
  if (tid < kBwdRows) {
    const int tl = tid / G;
    const int tok = qt0 + tl;
    if (tl < tpt && tok < tile.q_end) {
      const int head = tile.kvh * G + (tid - tl * G);
      const float2 rs = p.rowstat[(int64_t)tok * p.hq + head];
      r.l2 = rs.x;
      r.dl = rs.y;
      const int lim = visible_keys(p.toks[tok].P, tile.step, p.C, seq.c) - tile.u0;
      r.lim = lim < tile.nk ? lim : tile.nk;
    }
  }
  return r;
}

__device__ __forceinline__ void store_stats(QTileLds& s, const RowStats& r, int tid) {
  if (tid < kBwdRows) {
    s.l2[tid] = r.l2;
    s.dl[tid] = r.dl;
    s.lim[tid] = r.lim;
  }
}

}  // namespace

__global__ __launch_bounds__(kKvThreads, 1) void bwd_kv_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) QTileLds qs[2];

  const BwdTile tile = p.tiles[blockIdx.x];
  const SeqInfo seq = p.seqs[tile.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int qi = lane & 31;
  const int half = lane >> 5;
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  const int64_t key0 = (int64_t)seq.seg_off + tile.u0;  // first key row in the block

  const int tpt = kBwdRows / p.G;  // tokens per query tile
  const int ntiles = (tile.q_end - tile.q_begin + tpt - 1) / tpt;
  store_stats(qs[0], fetch_qtile(p, tile, seq, tile.q_begin, tid, qs[0]), tid);

  // this lane's key (column of S and dP): key 32*wave+qi, clamped to the tile
  const int my_key = 32 * wave + qi;
  const int kload = my_key < tile.nk ? my_key : tile.nk - 1;
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
    dk[nt] = f32x16{};
    dv[nt] = f32x16{};
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // ---- one query tile on LDS buffer B while tile it+1 is fetched into B^1
  auto step = [&](int it, auto buf_tag) {
    constexpr int B = decltype(buf_tag)::value;
    const QTileLds& cur = qs[B];
    const int qt0 = tile.q_begin + it * tpt;
    const bool more = it + 1 < ntiles;
    RowStats nst{0.f, 0.f, 0};
    if (more) nst = fetch_qtile(p, tile, seq, qt0 + tpt, tid, qs[B ^ 1]);
    const bool need_mask =
        qt0 < tile.q_full || qt0 + tpt > tile.q_end || tile.nk < kBwdKeys || tpt * p.G < kBwdRows;

    auto body = [&](auto mask_tag) {
      constexpr bool MASK = decltype(mask_tag)::value;
      // ---- S = Q K^T, dP = dO V^T (rows = queries, column = this lane's key)
      f32x16 s[2], dp[2];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        s[mt] = f32x16{};
        dp[mt] = f32x16{};
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          s[mt] = mfma32(ld16(&cur.q[tile_off<kBwdRows>(32 * mt + qi, 16 * c + 8 * half)]), kreg[c], s[mt]);
          dp[mt] = mfma32(ld16(&cur.g[tile_off<kBwdRows>(32 * mt + qi, 16 * c + 8 * half)]), vreg[c], dp[mt]);
        }
      }
      // phase fences: reads of a later phase hoisted over this one would
      // keep their results live across it and exhaust the registers
      __builtin_amdgcn_sched_barrier(0);
      // ---- P = exp2(S scale log2e - LSE log2e), dS = P (dP - Delta)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
          const int r0 = 32 * mt + 8 * vq + 4 * half;
          const float4 l4 = *reinterpret_cast<const float4*>(&cur.l2[r0]);
          const float4 d4 = *reinterpret_cast<const float4*>(&cur.dl[r0]);
          const int4 m4 = *reinterpret_cast<const int4*>(&cur.lim[r0]);
          const float lr[4] = {l4.x, l4.y, l4.z, l4.w};
          const float dr[4] = {d4.x, d4.y, d4.z, d4.w};
          const int mr[4] = {m4.x, m4.y, m4.z, m4.w};
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int v = 4 * vq + c;
            float pr = fast_exp2(__builtin_fmaf(s[mt][v], p.scale_log2, -lr[c]));
            if (MASK && my_key >= mr[c]) pr = 0.f;
            s[mt][v] = pr;
            dp[mt][v] = pr * (dp[mt][v] - dr[c]);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      // ---- dV += P^T dO, dK += dS^T Q.  k-block t covers query rows 16t..16t+15;
      // a lane of half h holds rows 16t+4h+{0..3} and 16t+8+4h+{0..3} of it, so
      // the dO / Q operand is read column-wise from the same rows.
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int v0 = 8 * (t & 1);
        const f32x16& ps = s[t >> 1];
        const f32x16& dss = dp[t >> 1];
        const bf16x8 pa =
            pack8(ps[v0], ps[v0 + 1], ps[v0 + 2], ps[v0 + 3], ps[v0 + 4], ps[v0 + 5], ps[v0 + 6], ps[v0 + 7]);
        const bf16x8 dsa = pack8(dss[v0], dss[v0 + 1], dss[v0 + 2], dss[v0 + 3], dss[v0 + 4], dss[v0 + 5],
                                 dss[v0 + 6], dss[v0 + 7]);
        const int ka = 16 * t + 4 * half, kb = ka + 8;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          dv[nt] = mfma32(pa, ld_tr8<kBwdRows>(cur.g, 32 * nt, ka, kb, lane), dv[nt]);
          dk[nt] = mfma32(dsa, ld_tr8<kBwdRows>(cur.q, 32 * nt, ka, kb, lane), dk[nt]);
        }
      }
    };
    if (need_mask) body(std::true_type{});
    else body(std::false_type{});

    if (more) store_stats(qs[B ^ 1], nst, tid);
    __builtin_amdgcn_s_waitcnt(0);  // this wavefront's direct loads have landed
    __syncthreads();
  };
  int it = 0;
  for (; it + 1 < ntiles; it += 2) {
    step(it, std::integral_constant<int, 0>{});
    step(it + 1, std::integral_constant<int, 1>{});
  }
  if (it < ntiles) step(it, std::integral_constant<int, 0>{});

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
// Query tile of 128 rows (4 wavefronts x 32), the same tiles as the forward.
// Accumulator layout: dQ^T, lane = one query row, rows = dims
// 32*dt + 8*(v/4) + 4*half + v%4.
template <int MODE>
__global__ __launch_bounds__(256, 2) void bwd_dq_kernel(BwdParams p) {
  // [buffer][K, V] plane tiles of 64 keys (see tile_off), double-buffered
  __shared__ __attribute__((aligned(16))) bf16 kvbuf[2][2][kFwdKeys * kHeadDim];

  const FwdTile tile = p.qtiles[blockIdx.x];
  const SeqInfo seq = p.seqs[tile.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int qi = lane & 31;
  const int half = lane >> 5;
  const int row = wave * 32 + qi;
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

  const int Pmin = p.toks[tile.tok_begin].P;
  const int Pmax = p.toks[tile.tok_begin + tile.ntok - 1].P;
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
  dim3 grid(p.num_qtiles), block(256);
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
