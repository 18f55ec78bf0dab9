// Forward branch attention for one context-parallel rank share (Sec. 3.2).
//
// One workgroup (4 wavefronts) owns a query tile of 128 rows: up to 128/G
// query tokens times the G query heads that share one KV head.  Each
// wavefront holds 32 rows.  Per ring step j the tile walks the visible prefix
// of rank j's KV block in 64-key tiles:
//   S^T = K Q^T       (bf16 MFMA 32x32x16, lane = one query row, so the row
//                      maximum is an in-register reduction plus one exchange
//                      with the other half-wavefront)
//   online softmax    (exp2 domain, fp32 statistics)
//   O^T += V^T P^T    (P^T taken straight from the S^T accumulator registers;
//                      V^T read column-wise from the row-major V tile with
//                      transposing LDS reads, in the matching key order)
// Tiles that are fully visible to every row skip the mask; the causal limit
// of a row in block j is a prefix of the block because positions increase
// with the local index (chunk j, then chunk 2C-1-j).  K and V tiles arrive by
// direct global-to-LDS loads, double-buffered across ring steps
// (walk_kv_tiles), so the next tile is in flight during the MFMAs.
//
// Epilogues
//   STEP  : merge the step's partial (O, LSE) into the running fp32 pair in
//           the workspace with Eq. lse-merge (first step writes it).
//   FINAL : read the running pair back as the main-sequence partial.
//   FUSED : all ring steps in one pass; the running pair stays in registers.
// FINAL and FUSED then compute the branch-local partial of every branch row
// (chain members 0..i, or the whole block; at most 64 keys, on the vector
// ALUs), merge it with the main partial by Eq. lse-merge and write bf16 O and
// the natural-log LSE.
#include <type_traits>

#include "ba_internal.h"
#include "device_common.h"
#include "kernels.h"

namespace ba {

namespace {

struct RowState {
  f32x16 o[4];  // O^T accumulator, d = 32*dt + 8*(v/4) + 4*half + v%4
  float m;      // running max (log2 domain)
  float l;      // running sum (this lane's keys only until the end)
};

}  // namespace

template <int MODE>
__global__ __launch_bounds__(256, 2) void fwd_kernel(FwdParams p) {
  // [buffer][K, V] plane tiles of 64 keys (see tile_off), double-buffered
  __shared__ __attribute__((aligned(16))) bf16 kvbuf[2][2][kFwdKeys * kHeadDim];

  const FwdTile tile = p.tiles[blockIdx.x];
  const SeqInfo seq = p.seqs[tile.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wavefront-uniform
  const int qi = lane & 31;
  const int half = lane >> 5;
  const int row = wave * 32 + qi;
  const int tl = row / p.G;
  const int head = tile.kvh * p.G + (row - tl * p.G);
  const bool valid = tl < tile.ntok;
  TokInfo tk;
  if (valid) tk = p.toks[tile.tok_begin + tl];
  else tk = TokInfo{0, -1, -1, -1};

  const bf16* qptr = tk.qrow >= 0 ? p.q_main + ((int64_t)tk.qrow * p.hq + head) * kHeadDim
                                  : p.q_br + ((int64_t)(-tk.qrow - 1) * p.hq + head) * kHeadDim;
  bf16x8 qreg[8];
#pragma unroll
  for (int ks8 = 0; ks8 < 8; ++ks8) {
    if (valid) qreg[ks8] = ld16(qptr + 16 * ks8 + 8 * half);
    else qreg[ks8] = bf16x8{};
  }

  RowState st;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) st.o[dt] = f32x16{};
  st.m = -INFINITY;
  st.l = 0.f;

  const int Pmin = p.toks[tile.tok_begin].P;
  const int Pmax = p.toks[tile.tok_begin + tile.ntok - 1].P;
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;

  if (MODE != kModeFinal) {
    // One 64-key tile: S^T = K Q^T, online softmax, O^T += V^T P^T.  MASK
    // (compile time) only on tiles crossing some row's causal limit.
    auto compute = [&](int j, int kv0, const bf16* ks, const bf16* vs, auto mask_tag) {
      constexpr bool MASK = decltype(mask_tag)::value;
      const int my_lim = valid ? visible_keys(tk.P, j, p.C, seq.c) : 0;
      // ---- S^T = K Q^T : two 32-key sub-tiles
      f32x16 s[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        s[kt] = f32x16{};
#pragma unroll
        for (int ks8 = 0; ks8 < 8; ++ks8)
          s[kt] = mfma32(ld16(&ks[tile_off<kFwdKeys>(32 * kt + qi, 16 * ks8 + 8 * half)]), qreg[ks8], s[kt]);
      }
      // ---- online softmax in the log2 domain; the scale is positive, so
      // the row maximum is taken on raw scores and applied once
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          if (MASK) {
            const int u = kv0 + 32 * kt + 8 * (v >> 2) + 4 * half + (v & 3);
            s[kt][v] = u < my_lim ? s[kt][v] : -INFINITY;
          }
          mx = fmaxf(mx, s[kt][v]);
        }
      }
      mx = fmaxf(mx, xor32(mx)) * p.scale_log2;
      const float m_new = fmaxf(st.m, mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = fast_exp2(st.m - m_use);
      float lsum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = fast_exp2(__builtin_fmaf(s[kt][v], p.scale_log2, -m_use));
          s[kt][v] = e;
          lsum += e;
        }
      }
      st.l = st.l * alpha + lsum;
      st.m = m_new;
      // the running output only needs rescaling when some row's maximum grew
      if (__ballot(alpha != 1.f)) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) st.o[dt] *= alpha;
      }
      // ---- O^T += V^T P^T : k-block t = keys 16t.. of the tile; a lane of
      // half h holds keys 16t+4h+{0..3} and 16t+8+4h+{0..3} of it in its S^T
      // registers, and reads the V^T operand from exactly those key rows
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const f32x16& src = s[t >> 1];
        const int v0 = 8 * (t & 1);
        const bf16x8 pb = pack8(src[v0], src[v0 + 1], src[v0 + 2], src[v0 + 3], src[v0 + 4], src[v0 + 5],
                                src[v0 + 6], src[v0 + 7]);
        const int ka = 16 * t + 4 * half, kb = ka + 8;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
          st.o[dt] = mfma32(ld_tr8<kFwdKeys>(vs, 32 * dt, ka, kb, lane), pb, st.o[dt]);
      }
    };
    walk_kv_tiles(p, seq, tile.kvh, Pmax, wave, lane, kvbuf, [&](int j, int kv0, const bf16* ks, const bf16* vs) {
      if (kv0 + kFwdKeys <= visible_keys(Pmin, j, p.C, seq.c)) compute(j, kv0, ks, vs, std::false_type{});
      else compute(j, kv0, ks, vs, std::true_type{});
    });
  }

  // ------------------------------------------------------------ epilogues
  const int64_t acc_row = (int64_t)(tile.tok_begin + tl) * p.hq + head;

  if (MODE == kModeStep) {
    const float l_tot = st.l + xor32(st.l);
    if (!valid) return;
    float* oacc = p.o_acc + acc_row * kHeadDim;
    if (l_tot > 0.f) {
      const float lse2 = st.m + __log2f(l_tot);
      const float inv = 1.f / l_tot;
      float wa = 0.f, wb = inv;
      float lse_new = lse2;
      if (!p.acc_first) {
        const float la = p.lse_acc[acc_row];
        const float hi = fmaxf(la, lse2);
        const float ea = fast_exp2(la - hi);  // la = -inf gives 0
        const float eb = fast_exp2(lse2 - hi);
        const float tot = ea + eb;
        lse_new = hi + __log2f(tot);
        wa = ea / tot;
        wb = eb / tot * inv;
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
          float4* dst = reinterpret_cast<float4*>(oacc + 32 * dt + 8 * vq + 4 * half);
          float4 prev = make_float4(0.f, 0.f, 0.f, 0.f);
          if (!p.acc_first) prev = *dst;
          float4 o;
          o.x = wa * prev.x + wb * st.o[dt][4 * vq + 0];
          o.y = wa * prev.y + wb * st.o[dt][4 * vq + 1];
          o.z = wa * prev.z + wb * st.o[dt][4 * vq + 2];
          o.w = wa * prev.w + wb * st.o[dt][4 * vq + 3];
          *dst = o;
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

  // main-sequence partial: normalised output in st.o, LSE (log2) in lse_m
  float lse_m;
  if (MODE == kModeFinal) {
    if (valid) {
      const float* oacc = p.o_acc + acc_row * kHeadDim;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
          const float4 a = *reinterpret_cast<const float4*>(oacc + 32 * dt + 8 * vq + 4 * half);
          st.o[dt][4 * vq + 0] = a.x;
          st.o[dt][4 * vq + 1] = a.y;
          st.o[dt][4 * vq + 2] = a.z;
          st.o[dt][4 * vq + 3] = a.w;
        }
      lse_m = p.lse_acc[acc_row];
    } else {
      lse_m = -INFINITY;
    }
  } else {
    const float l_tot = st.l + xor32(st.l);
    if (l_tot > 0.f) {
      lse_m = st.m + __log2f(l_tot);
      const float inv = 1.f / l_tot;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) st.o[dt] *= inv;
    } else {
      lse_m = -INFINITY;
    }
  }

  // ---- branch-local partial (vector ALUs; at most 64 keys per row)
  int nb = 0;
  GroupInfo gi{0, 1, 0, 0};
  if (valid && tk.grp >= 0) {
    gi = p.groups[tk.grp];
    nb = gi.kind == BA_KIND_EAGLE_CHAIN ? tk.gidx + 1 : gi.len;
  }
  float mb = -INFINITY, lb = 0.f;
  f32x16 ob[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) ob[dt] = f32x16{};
  for (int b = 0; b < BA_MAX_GROUP_LEN; ++b) {
    const bool active = b < nb;
    if (__ballot(active) == 0) break;
    const int64_t krow = (int64_t)gi.row0 + (int64_t)b * gi.stride;
    const bf16* kb = p.k_br + krow * kv_row_stride + tile.kvh * kHeadDim;
    const bf16* vb = p.v_br + krow * kv_row_stride + tile.kvh * kHeadDim;
    float dot = 0.f;
    if (active) {
#pragma unroll
      for (int ks8 = 0; ks8 < 8; ++ks8) {
        const bf16x8 kv = ld16(kb + 16 * ks8 + 8 * half);
#pragma unroll
        for (int e = 0; e < 8; ++e) dot += (float)qreg[ks8][e] * (float)kv[e];
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
  if (!valid) return;

  // ---- Eq. lse-merge of the main and branch partials, then write out
  const float lse_b = lb > 0.f ? mb + __log2f(lb) : -INFINITY;
  const float hi = fmaxf(lse_m, lse_b);
  const float wm = lse_m == -INFINITY ? 0.f : fast_exp2(lse_m - hi);
  const float wbr = lse_b == -INFINITY ? 0.f : fast_exp2(lse_b - hi);
  const float tot = wm + wbr;
  const float lse2 = hi + __log2f(tot);
  const float cm = wm / tot;
  const float cb = lb > 0.f ? wbr / (tot * lb) : 0.f;

  bf16* out;
  float* lse_out;
  if (tk.qrow >= 0) {
    out = p.o_main + ((int64_t)tk.qrow * p.hq + head) * kHeadDim;
    lse_out = p.lse_main + (int64_t)head * p.n_local + tk.qrow;
  } else {
    const int64_t br = -tk.qrow - 1;
    out = p.o_br + (br * p.hq + head) * kHeadDim;
    lse_out = p.lse_br + (int64_t)head * p.n_br + br;
  }
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int vq = 0; vq < 4; ++vq) {
      const int v = 4 * vq;
      *reinterpret_cast<bf16x4*>(out + 32 * dt + 8 * vq + 4 * half) =
          pack4(cm * st.o[dt][v] + cb * ob[dt][v], cm * st.o[dt][v + 1] + cb * ob[dt][v + 1],
                cm * st.o[dt][v + 2] + cb * ob[dt][v + 2], cm * st.o[dt][v + 3] + cb * ob[dt][v + 3]);
    }
  if (half == 0) *lse_out = lse2 * kLn2;
}

hipError_t launch_fwd(const FwdParams& p, int mode, hipStream_t stream) {
  if (p.num_tiles == 0) return hipSuccess;
  dim3 grid(p.num_tiles), block(256);
  if (mode == kModeStep) hipLaunchKernelGGL(fwd_kernel<kModeStep>, grid, block, 0, stream, p);
  else if (mode == kModeFinal) hipLaunchKernelGGL(fwd_kernel<kModeFinal>, grid, block, 0, stream, p);
  else hipLaunchKernelGGL(fwd_kernel<kModeFused>, grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace ba
