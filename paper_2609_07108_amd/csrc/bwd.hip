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
//                LDS with register prefetch.  No atomics.
//   dq         : dQ, query-tile parallel like the forward: per key tile
//                S^T = K Q^T, dP^T = V dO^T, dS^T, dQ^T += K^T dS^T, with the
//                branch-local keys handled in the epilogue.  Splitting dQ off
//                costs two extra contractions but avoids fp32 atomics, whose
//                throughput (about one 4-byte update per L2 channel and clock)
//                would otherwise bound the whole backward.
//   branch     : dK and dV of the branch-local keys (at most 64 per group).
#include "ba_internal.h"
#include "device_common.h"
#include "kernels.h"

namespace ba {

namespace {

constexpr int kRowStride = kHeadDim + 8;  // padded row-major [rows][d] LDS tiles

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
// Workgroup of 8 wavefronts (2 per SIMD) on 128 keys: wavefront w owns keys
// 32*(w%4).. and the query rows 32*(w/4).. of every 64-row tile, so each key
// group is covered by two wavefronts whose dK/dV partial sums are added
// through LDS at the end.  The K and V tiles stay in LDS for the whole walk
// (B operands of S = Q K^T and dP = dO V^T); the query tiles are
// double-buffered in LDS and prefetched through registers.
namespace {

constexpr int kKvWaves = 8;
constexpr int kKvThreads = 64 * kKvWaves;

struct QTileLds {
  bf16 q[kBwdRows * kRowStride];
  bf16 g[kBwdRows * kRowStride];
  float l2[kBwdRows];
  float dl[kBwdRows];
  int lim[kBwdRows];
};

struct KvLds {
  union {
    QTileLds qs[2];
    float red[4 * 64 * 64];  // end-of-kernel exchange of one accumulator set
  };
  bf16 k[kBwdKeys * kRowStride];
  bf16 v[kBwdKeys * kRowStride];
};

// One thread's share of the next query tile: threads 0..255 load 4 rows x 8
// dims of Q, threads 256..511 the same of dO; threads 0..63 also load the row
// statistics and the visible-key limit.
struct QTileRegs {
  bf16x8 x[4];
  float l2, dl;
  int lim;
};

__device__ __forceinline__ void load_qtile(const BwdParams& p, const BwdTile& tile, const SeqInfo& seq,
                                           int qt0, int tid, QTileRegs& r) {
  const int G = p.G;
  const int tpt = kBwdRows / G;  // rows past tpt*G belong to no token
  const int t = tid & 255;
  const bool is_do = tid >= 256;
  const int rg = t >> 4, dc = t & 15;  // rows 4rg..4rg+3, dims 8dc..8dc+7
#pragma unroll
  for (int r4 = 0; r4 < 4; ++r4) {
    const int row = 4 * rg + r4;
    const int tl = row / G;
    const int tok = qt0 + tl;
    if (tl < tpt && tok < tile.q_end) {
      const TokInfo tk = p.toks[tok];
      const int head = tile.kvh * G + (row - tl * G);
      r.x[r4] = ld16(row_ptr(is_do ? p.do_main : p.q_main, is_do ? p.do_br : p.q_br, tk.qrow, p.hq, head) +
                     8 * dc);
    } else {
      r.x[r4] = bf16x8{};
    }
  }
  r.l2 = 0.f;
  r.dl = 0.f;
  r.lim = 0;
  if (tid < kBwdRows) {
    const int tl = tid / G;
    const int tok = qt0 + tl;
    if (tl < tpt && tok < tile.q_end) {
      const int head = tile.kvh * G + (tid - tl * G);
      const float2 rs = p.rowstat[(int64_t)tok * p.hq + head];
      r.l2 = rs.x;
      r.dl = rs.y;
      int lim = visible_keys(p.toks[tok].P, tile.step, p.C, seq.c) - tile.u0;
      r.lim = lim < tile.nk ? lim : tile.nk;
    }
  }
}

__device__ __forceinline__ void store_qtile(QTileLds& s, const QTileRegs& r, int tid) {
  const int t = tid & 255;
  const int rg = t >> 4, dc = t & 15;
  bf16* dst = tid >= 256 ? s.g : s.q;
#pragma unroll
  for (int r4 = 0; r4 < 4; ++r4) st16(&dst[(4 * rg + r4) * kRowStride + 8 * dc], r.x[r4]);
  if (tid < kBwdRows) {
    s.l2[tid] = r.l2;
    s.dl[tid] = r.dl;
    s.lim[tid] = r.lim;
  }
}

}  // namespace

__global__ __launch_bounds__(kKvThreads, 1) void bwd_kv_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) KvLds sm;

  const BwdTile tile = p.tiles[blockIdx.x];
  const SeqInfo seq = p.seqs[tile.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int kw = wave & 3;   // key group
  const int rh = wave >> 2;  // row half of every query tile
  const int qi = lane & 31;
  const int half = lane >> 5;
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  const int64_t key0 = (int64_t)seq.seg_off + tile.u0;  // first key row in the block
  const bf16* kbase = p.k_step[tile.step] + key0 * kv_row_stride + tile.kvh * kHeadDim;
  const bf16* vbase = p.v_step[tile.step] + key0 * kv_row_stride + tile.kvh * kHeadDim;

  // this lane's key (column of S and dP): key 32*kw+qi of the tile
  const int my_key = 32 * kw + qi;
  {
    const int kk = tid >> 2, qq = tid & 3;  // K and V tiles: key kk, dims 32qq..32qq+31
    const int u = kk < tile.nk ? kk : tile.nk - 1;
    const bf16* ksrc = kbase + (int64_t)u * kv_row_stride + 32 * qq;
    const bf16* vsrc = vbase + (int64_t)u * kv_row_stride + 32 * qq;
#pragma unroll
    for (int c8 = 0; c8 < 4; ++c8) {
      st16(&sm.k[kk * kRowStride + 32 * qq + 8 * c8], ld16(ksrc + 8 * c8));
      st16(&sm.v[kk * kRowStride + 32 * qq + 8 * c8], ld16(vsrc + 8 * c8));
    }
  }

  f32x16 dk[4], dv[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    dk[nt] = f32x16{};
    dv[nt] = f32x16{};
  }

  const int tpt = kBwdRows / p.G;  // tokens per query tile
  const int ntiles = (tile.q_end - tile.q_begin + tpt - 1) / tpt;
  {
    QTileRegs r;
    load_qtile(p, tile, seq, tile.q_begin, tid, r);
    store_qtile(sm.qs[0], r, tid);
  }
  __syncthreads();

  const int r0w = 32 * rh;  // first query row of this wavefront inside a tile
  for (int it = 0; it < ntiles; ++it) {
    const int qt0 = tile.q_begin + it * tpt;
    const QTileLds& cur = sm.qs[it & 1];
    const bool more = it + 1 < ntiles;
    QTileRegs nxt;
    if (more) load_qtile(p, tile, seq, qt0 + tpt, tid, nxt);  // in flight during the MFMAs below
    const bool need_mask =
        qt0 < tile.q_full || qt0 + tpt > tile.q_end || tile.nk < kBwdKeys || tpt * p.G < kBwdRows;

    // ---- S = Q K^T, dP = dO V^T (rows = this wavefront's 32 queries, column = the lane's key)
    f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      s = mfma32(ld16(&cur.q[(r0w + qi) * kRowStride + 16 * c + 8 * half]),
                 ld16(&sm.k[my_key * kRowStride + 16 * c + 8 * half]), s);
      dp = mfma32(ld16(&cur.g[(r0w + qi) * kRowStride + 16 * c + 8 * half]),
                  ld16(&sm.v[my_key * kRowStride + 16 * c + 8 * half]), dp);
    }
    // ---- P = exp2(S scale log2e - LSE log2e), dS = P (dP - Delta)
#pragma unroll
    for (int vq = 0; vq < 4; ++vq) {
      const int r0 = r0w + 8 * vq + 4 * half;
      const float4 l4 = *reinterpret_cast<const float4*>(&cur.l2[r0]);
      const float4 d4 = *reinterpret_cast<const float4*>(&cur.dl[r0]);
      const int4 m4 = *reinterpret_cast<const int4*>(&cur.lim[r0]);
      const float lr[4] = {l4.x, l4.y, l4.z, l4.w};
      const float dr[4] = {d4.x, d4.y, d4.z, d4.w};
      const int mr[4] = {m4.x, m4.y, m4.z, m4.w};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int v = 4 * vq + c;
        float pr = fast_exp2(s[v] * p.scale_log2 - lr[c]);
        if (need_mask && my_key >= mr[c]) pr = 0.f;
        s[v] = pr;
        dp[v] = pr * (dp[v] - dr[c]);
      }
    }
    // ---- dV += P^T dO, dK += dS^T Q.  k-block t covers rows r0w+16t..+15; a
    // lane of half h holds rows 16t+4h+{0..3} and 16t+8+4h+{0..3} of it, so
    // the dO / Q operand is read column-wise from the same rows.
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int v0 = 8 * t;
      const bf16x8 pa = pack8(s[v0], s[v0 + 1], s[v0 + 2], s[v0 + 3], s[v0 + 4], s[v0 + 5], s[v0 + 6], s[v0 + 7]);
      const bf16x8 dsa =
          pack8(dp[v0], dp[v0 + 1], dp[v0 + 2], dp[v0 + 3], dp[v0 + 4], dp[v0 + 5], dp[v0 + 6], dp[v0 + 7]);
      const int ka = r0w + 16 * t + 4 * half, kb = ka + 8;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        dv[nt] = mfma32(pa, ld_tr8(cur.g, kRowStride, 32 * nt, ka, kb, lane), dv[nt]);
        dk[nt] = mfma32(dsa, ld_tr8(cur.q, kRowStride, 32 * nt, ka, kb, lane), dk[nt]);
      }
    }
    if (more) store_qtile(sm.qs[(it + 1) & 1], nxt, tid);
    __syncthreads();
  }

  // ---- add the two row halves' partial sums (wavefronts w and w+4), one
  // accumulator set at a time through the (now idle) query-tile buffers
  float* red = sm.red + (kw * 64) * 64;
  if (rh == 1) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int v = 0; v < 16; ++v) red[(16 * nt + v) * 64 + lane] = dk[nt][v];
  }
  __syncthreads();
  if (rh == 0) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int v = 0; v < 16; ++v) dk[nt][v] += red[(16 * nt + v) * 64 + lane];
  }
  __syncthreads();
  if (rh == 1) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int v = 0; v < 16; ++v) red[(16 * nt + v) * 64 + lane] = dv[nt][v];
  }
  __syncthreads();
  if (rh == 1) return;
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int v = 0; v < 16; ++v) dv[nt][v] += red[(16 * nt + v) * 64 + lane];

  // ---- write dK (scaled) and dV: accumulator column = dim, rows = keys
  void* dkout = p.dk_step[tile.step];
  void* dvout = p.dv_step[tile.step];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int key = 32 * kw + 8 * (v >> 2) + 4 * half + (v & 3);
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
  __shared__ __attribute__((aligned(16))) bf16 ks[kFwdKeys * kRowStride];
  __shared__ __attribute__((aligned(16))) bf16 vs[kFwdKeys * kRowStride];

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
    for (int i = p.step_first; i < p.step_first + p.step_count; ++i) {
      const int j = ((p.rank - i) % p.C + p.C) % p.C;
      const int lim_lo = visible_keys(Pmin, j, p.C, seq.c);
      const int lim_hi = visible_keys(Pmax, j, p.C, seq.c);
      const int my_lim = valid ? visible_keys(tk.P, j, p.C, seq.c) : 0;
      const bf16* kbase = p.k_step[j] + (int64_t)seq.seg_off * kv_row_stride + tile.kvh * kHeadDim;
      const bf16* vbase = p.v_step[j] + (int64_t)seq.seg_off * kv_row_stride + tile.kvh * kHeadDim;
      for (int kv0 = 0; kv0 < lim_hi; kv0 += kFwdKeys) {
        {
          const int kk = tid >> 2, qq = tid & 3;
          int u = kv0 + kk;
          u = u < lim_hi ? u : lim_hi - 1;
          const bf16* ksrc = kbase + (int64_t)u * kv_row_stride + 32 * qq;
          const bf16* vsrc = vbase + (int64_t)u * kv_row_stride + 32 * qq;
#pragma unroll
          for (int c8 = 0; c8 < 4; ++c8) {
            st16(&ks[kk * kRowStride + 32 * qq + 8 * c8], ld16(ksrc + 8 * c8));
            st16(&vs[kk * kRowStride + 32 * qq + 8 * c8], ld16(vsrc + 8 * c8));
          }
        }
        __syncthreads();
        // ---- S^T = K Q^T and dP^T = V dO^T (two 32-key sub-tiles)
        f32x16 s[2], dp[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          s[kt] = f32x16{};
          dp[kt] = f32x16{};
#pragma unroll
          for (int c = 0; c < 8; ++c) {
            s[kt] = mfma32(ld16(&ks[(32 * kt + qi) * kRowStride + 16 * c + 8 * half]), qreg[c], s[kt]);
            dp[kt] = mfma32(ld16(&vs[(32 * kt + qi) * kRowStride + 16 * c + 8 * half]), greg[c], dp[kt]);
          }
        }
        // ---- dS^T = P^T (dP^T - Delta), P^T = exp2(S^T scale log2e - LSE log2e)
        const bool need_mask = kv0 + kFwdKeys > lim_lo;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            float pr = fast_exp2(s[kt][v] * p.scale_log2 - lse2);
            if (need_mask) {
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
          const int ka = 16 * t + 4 * half, kb = 16 * t + 8 + 4 * half;
#pragma unroll
          for (int dt = 0; dt < 4; ++dt) dq[dt] = mfma32(ld_tr8(ks, kRowStride, 32 * dt, ka, kb, lane), b, dq[dt]);
        }
        __syncthreads();
      }
    }
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
