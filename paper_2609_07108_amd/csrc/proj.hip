// Grouped-query QKV projection of a draft layer's attention input, with the
// rotary embedding of the queries and keys applied in the projection's
// epilogue, and its backward.  This is the step in front of branch attention
// inside a draft layer.  The paper gives no projection detail; this library
// reads the draft layer as a Llama-style decoder layer (its own reading):
// hidden states are projected to q-heads and fewer kv-heads, queries and keys
// rotated by their positions, then attended.
//
//   forward:  Y = X W^T, X [rows, hidden], W [(hq + 2 hkv) * 128, hidden]
//             (the fused q/k/v weight of a linear layer, output-major);
//             Y's 128-column head blocks are the q-heads, then the k-heads,
//             then the v-heads; q and k rotated by pos[row] (dims j, j + 64
//             by the angle pos * theta^(-j/64)), all three written as bf16
//             [rows, heads, 128].
//   backward: dY = [R^T dQ, R^T dK, dV] (bf16, in the workspace), then
//             dX = dY W and dW = dY^T X (fp32 accumulation).
//
// One GEMM kernel serves all three products.  C[i][j] = sum_k A(i,k) B(j,k)
// over 128 x 128 output tiles, 64 reduction values per stage, two stages of
// LDS; each operand is either stored with its reduction index contiguous
// ([i][k], "k-major") or with its row index contiguous ([k][i], "i-major").
// A workgroup of four wavefronts computes one tile, each wavefront a 64 x 64
// quarter as 2 x 2 v_mfma_f32_32x32x16_bf16 accumulators.  Operands move
// global -> registers -> LDS through two register sets, so the loads of
// stage t+2 are in flight during the MFMAs of stage t.
#include <cmath>
#include <string>

#include "ba_internal.h"
#include "device_common.h"
#include "kernels.h"

namespace ba {
namespace {

constexpr int kTile = 128;               // output tile rows and columns
constexpr int kBk = 64;                  // reduction values per stage
constexpr int kOpElems = kTile * kBk;    // one operand tile, bf16 elements (16 KB)
constexpr int kStageLd = kTile + 8;      // fp32 staging row pitch of the epilogue (conflict-free writes)
constexpr int kSmemBytes = (4 * kOpElems * 2 > kTile * kStageLd * 4) ? 4 * kOpElems * 2 : kTile * kStageLd * 4;

// k-major operand tile: 128 rows x 64 reduction values, 128 B per row; the
// eight 16-byte chunks of row r are XOR-permuted by (r/2) % 8, so that the
// 16 lanes of an MFMA operand read (16 consecutive rows, one chunk) and of a
// tile store (two rows, eight chunks) touch 16 distinct 16-byte bank groups.
// i-major operand tile: 64 reduction rows x 128 columns as a plane tile
// (tile_off), read with transposed 8-byte reads.
__device__ __forceinline__ int kmaj_off(int r, int chunk) { return r * kBk + ((chunk ^ ((r >> 1) & 7)) << 3); }

// Per-lane LDS byte offsets inside one operand tile, computed once: every
// operand read, transposed read and tile store of the main loop is one of
// these plus a compile-time constant (the instruction's offset field takes
// it for row reads and stores; transposed reads still pay one add each),
// since the XOR terms of both layouts depend on the lane alone.
//   operand of rows r0.. (r0 % 32 == 0) at reduction step ks:
//     k-major: rd[ks] + 128 r0;  i-major: tlo / thi + 1024 ks + 128 r0
//   store of fetch q: st + 4096 q (k-major) or st + 1024 q (i-major)
template <bool kIMajor>
struct LaneOfs {
  uint32_t rd[4], tlo, thi, st;
  __device__ __forceinline__ explicit LaneOfs(int tid) {
    const int lane = tid & 63, h = lane >> 5;
    if constexpr (!kIMajor) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) rd[ks] = 2u * (uint32_t)kmaj_off(lane & 31, 2 * ks + h);
      tlo = thi = 0;
      st = 2u * (uint32_t)kmaj_off(tid >> 3, tid & 7);
    } else {
      const int i = lane & 15, col = (lane & 16) + 4 * (i & 3);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) rd[ks] = 0;
      tlo = 2u * (uint32_t)tile_off<kBk>(8 * h + (i >> 2), col);
      thi = 2u * (uint32_t)tile_off<kBk>(8 * h + 4 + (i >> 2), col);
      st = 2u * (uint32_t)tile_off<kBk>(tid >> 4, 8 * (tid & 15));
    }
  }
};

template <bool kIMajor, int kR0, int kKs>
__device__ __forceinline__ bf16x8 operand(uint32_t tile, const LaneOfs<kIMajor>& o) {
  if constexpr (!kIMajor) {
    return lds_ld16(tile + o.rd[kKs] + 128u * kR0);
  } else {
    const uint32_t c = 1024u * kKs + 128u * kR0;
    const bf16x4 lo = lds_ld_tr4(tile + o.tlo + c), hi = lds_ld_tr4(tile + o.thi + c);
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  }
}

template <bool kIMajor>
__device__ __forceinline__ void store_tile(uint32_t tile, const LaneOfs<kIMajor>& o, const bf16x8 (&g)[4]) {
#pragma unroll
  for (int q = 0; q < 4; ++q)
    *(__attribute__((address_space(3))) bf16x8*)(uintptr_t)(tile + o.st + (kIMajor ? 1024u : 4096u) * q) = g[q];
}

// Global side of one operand: per-lane 32-bit byte offsets from a
// wave-uniform base that advances by one stage per iteration.
// k-major ([i][k], ld elements per row): thread t fetches chunk t % 8 of
// tile rows t/8 + 32q; rows past the end re-read the last row (their results
// are never stored); stage kt starts at base + i0 ld + 64 kt.  The
// reduction slices lie inside K (K % 64 == 0).
// i-major ([k][i]): thread t fetches columns 8 (t % 16) .. +7 of reduction
// rows t/16 + 16q; stage kt starts at base + 64 kt ld + i0.  Rows at or
// past K (a ragged last stage only) read row K-1 and become zeros.
template <bool kIMajor>
struct Fetch {
  const char* base;  // stage 0
  int64_t stage;     // bytes per stage
  uint32_t off[4];
  __device__ __forceinline__ Fetch(const bf16* a, int64_t ld, int64_t i0, int64_t ni, int tid) {
    if constexpr (!kIMajor) {
      base = reinterpret_cast<const char*>(a + i0 * ld);
      stage = 2 * kBk;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int64_t r = i0 + (tid >> 3) + 32 * q;
        r = (r < ni ? r : ni - 1) - i0;
        off[q] = (uint32_t)(2 * (r * ld + 8 * (tid & 7)));
      }
    } else {
      base = reinterpret_cast<const char*>(a + i0);
      stage = 2 * kBk * ld;
#pragma unroll
      for (int q = 0; q < 4; ++q) off[q] = (uint32_t)(2 * (((tid >> 4) + 16 * q) * ld + 8 * (tid & 15)));
    }
  }
  __device__ __forceinline__ void load(int64_t kt, bf16x8 (&g)[4]) const {
    const char* b = base + kt * stage;
#pragma unroll
    for (int q = 0; q < 4; ++q) g[q] = *reinterpret_cast<const bf16x8*>(b + off[q]);
  }
  // i-major only: the last stage when it reaches past K
  __device__ __forceinline__ void load_tail(int64_t kt, int64_t K, int64_t ld, int tid, bf16x8 (&g)[4]) const {
    const char* b = base + kt * stage;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t kk = kt * kBk + (tid >> 4) + 16 * q;
      const int64_t back = kk < K ? 0 : kk - (K - 1);  // rows to step back to reach row K-1
      const bf16x8 v = *reinterpret_cast<const bf16x8*>(b + off[q] - 2 * back * ld);
      g[q] = kk < K ? v : bf16x8{};
    }
  }
};

}  // namespace

// C = A B^T over one 128 x 128 tile per workgroup; see the file comment.
template <bool kAI, bool kBI, int kEpi>
__global__ __launch_bounds__(256, 2) void proj_gemm_kernel(const ProjGemmParams p) {
  __shared__ __align__(16) unsigned char smem_raw[kSmemBytes];
  bf16* smem = reinterpret_cast<bf16*>(smem_raw);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_j = p.J / kTile;
  const int64_t ti = blockIdx.x / tiles_j;
  const int tj = (int)(blockIdx.x - ti * tiles_j);
  const int64_t i0 = ti * kTile;
  const int j0 = tj * kTile;
  const int64_t nk = (p.K + kBk - 1) / kBk;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  const LaneOfs<kAI> oa(tid);
  const LaneOfs<kBI> ob(tid);
  const Fetch<kAI> fa(p.a, p.lda, i0, p.I, tid);
  const Fetch<kBI> fb(p.b, p.ldb, j0, p.J, tid);
  const uint32_t lds0 = lds_addr(smem);
  constexpr uint32_t kOpBytes = 2u * kOpElems;
  // the stage that reaches past a ragged reduction end (i-major operands only)
  const int64_t tail = (p.K % kBk) ? nk - 1 : nk;
  auto fetch = [&](int64_t kt, bf16x8 (&ga)[4], bf16x8 (&gb)[4]) {
    if (kt != tail) {
      fa.load(kt, ga);
      fb.load(kt, gb);
    } else {
      if constexpr (kAI) fa.load_tail(kt, p.K, p.lda, tid, ga); else fa.load(kt, ga);
      if constexpr (kBI) fb.load_tail(kt, p.K, p.ldb, tid, gb); else fb.load(kt, gb);
    }
  };

  // Two register sets: while stage t is multiplied, the loads of stage
  // t + 2 are in flight into one set and the other set (stage t + 1, loaded
  // during the previous stage) is written to the free LDS buffer afterwards,
  // so every load has two stages of MFMA work to arrive.
  bf16x8 ga0[4], gb0[4], ga1[4], gb1[4];
  if (nk > 0) {
    fetch(0, ga0, gb0);
    store_tile<kAI>(lds0, oa, ga0);
    store_tile<kBI>(lds0 + kOpBytes, ob, gb0);
    __syncthreads();
  }
  // The fetches are unconditional (past the end they re-read the last stage,
  // which is never stored): with a skipped fetch on some path, the compiler's
  // wait counts at the stores would have to cover the newer loads as well.
  if (nk > 0) fetch(nk > 1 ? 1 : 0, ga1, gb1);
  auto iterate = [&](int64_t kt, const bf16x8 (&ca)[4], const bf16x8 (&cb)[4], bf16x8 (&na)[4],
                     bf16x8 (&nb)[4]) {
    fetch(kt + 2 < nk ? kt + 2 : nk - 1, na, nb);
    const uint32_t TA = lds0 + (uint32_t)(kt & 1) * 2u * kOpBytes;
    const uint32_t TB = TA + kOpBytes;
    static_for<kBk / 16>([&](auto ks) {
      constexpr int kKs = decltype(ks)::value;
      const bf16x8 a0 = operand<kAI, 0, kKs>(TA + 128u * 64 * wm, oa);
      const bf16x8 a1 = operand<kAI, 32, kKs>(TA + 128u * 64 * wm, oa);
      const bf16x8 b0 = operand<kBI, 0, kKs>(TB + 128u * 64 * wn, ob);
      const bf16x8 b1 = operand<kBI, 32, kKs>(TB + 128u * 64 * wn, ob);
      acc[0][0] = mfma32(a0, b0, acc[0][0]);
      acc[0][1] = mfma32(a0, b1, acc[0][1]);
      acc[1][0] = mfma32(a1, b0, acc[1][0]);
      acc[1][1] = mfma32(a1, b1, acc[1][1]);
    });
    if (kt + 1 < nk) {
      const uint32_t nxt = lds0 + (uint32_t)((kt + 1) & 1) * 2u * kOpBytes;
      store_tile<kAI>(nxt, oa, ca);
      store_tile<kBI>(nxt + kOpBytes, ob, cb);
    }
    __syncthreads();
  };
  for (int64_t kt = 0; kt < nk; kt += 2) {
    iterate(kt, ga1, gb1, ga0, gb0);
    if (kt + 1 < nk) iterate(kt + 1, ga0, gb0, ga1, gb1);
  }

  // accumulator element v of lane l: row 8 (v/4) + 4 (l/32) + v%4, column l%32
  if constexpr (kEpi == kProjEpiPlain) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int64_t row = i0 + 64 * wm + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
          const int64_t col = j0 + 64 * wn + 32 * j + (lane & 31);
          if (row < p.I) {
            const int64_t at = row * p.ldc + col;
            if (p.c_f32) {
              float* c = static_cast<float*>(p.c);
              c[at] = p.accumulate ? c[at] + acc[i][j][v] : acc[i][j][v];
            } else {
              static_cast<bf16*>(p.c)[at] = (bf16)acc[i][j][v];
            }
          }
        }
  } else {
    // stage the tile (one head of 128 columns) in LDS, then one 16-lane row
    // per output row: lane l16 holds dims 8 l16 .. +7, its rotation partner
    // (dims +-64) sits in lane l16 ^ 8 of the same DPP row.
    float* S = reinterpret_cast<float*>(smem_raw);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          S[(64 * wm + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * kStageLd + 64 * wn + 32 * j +
            (lane & 31)] = acc[i][j][v];
    __syncthreads();
    const int head = tj;
    bf16* dst;
    int hh, nh;
    if (head < p.hq) {
      dst = p.q; hh = head; nh = p.hq;
    } else if (head < p.hq + p.hkv) {
      dst = p.k; hh = head - p.hq; nh = p.hkv;
    } else {
      dst = p.v; hh = head - p.hq - p.hkv; nh = p.hkv;
    }
    const bool rot = p.rotate && head < p.hq + p.hkv;
    const int l16 = tid & 15, grp = tid >> 4;
    const float sg = l16 < 8 ? -1.f : 1.f;
    RopeFreq f[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = rot ? p.freq.f[8 * (l16 & 7) + e] : RopeFreq{0.f, 0.f};
#pragma unroll 2
    for (int rr = 0; rr < kTile / 16; ++rr) {
      const int r = grp + 16 * rr;
      const int64_t row = i0 + r;
      const float4 x0 = *reinterpret_cast<const float4*>(S + r * kStageLd + 8 * l16);
      const float4 x1 = *reinterpret_cast<const float4*>(S + r * kStageLd + 8 * l16 + 4);
      const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
      const int ps = (rot && row < p.I) ? p.pos[row] : -1;
      float y[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float sn = 0.f, cs = 1.f;
        if (ps >= 0) rope_sincos_fast(ps, f[e], sn, cs);
        const float xp = dpp_mov<0x128>(x[e]);  // row_ror:8, the partner lane l16 ^ 8
        y[e] = fmaf(xp, sn * sg, x[e] * cs);
      }
      if (row < p.I) st16(dst + (row * nh + hh) * kHeadDim + 8 * l16, pack8(y[0], y[1], y[2], y[3], y[4], y[5], y[6], y[7]));
    }
  }
}

// ------------------------------------------------------------------ wide
// The same products on 256 x 256 output tiles when K % 64 == 0: eight
// wavefronts (two per SIMD), wavefront w computing the 128 x 64 block at
// rows 128 (w / 4), columns 64 (w % 4) as 4 x 2 MFMA accumulators, so each
// k-step's six operand fragments (6 KB) feed eight MFMAs (0.75 KB of LDS
// reads per MFMA against 1 KB for the 64 x 64 blocks above).  Operands go
// global -> LDS by direct loads (no register staging, no LDS store
// instructions) into two stages of 64 reduction values, one barrier per
// stage.  Four wavefronts of 128 x 128 (0.5 KB per MFMA, one per SIMD)
// measured slower.
namespace {

constexpr int kWTile = 256;                          // output tile rows and columns
constexpr int kWBk = 64;                             // reduction values per stage
constexpr int kWStages = 2;
constexpr int kWKsteps = kWBk / 16;                  // MFMA k-steps per stage
constexpr uint32_t kWOpBytes = kWTile * kWBk * 2;    // one operand of one stage (32 KB)
constexpr int kWPieces = (int)(kWOpBytes / 1024 / 4);  // 1 KB direct loads per wavefront and stage
constexpr int kWRows = 128;                          // epilogue rows staged per pass
constexpr int kWStageLd = kWTile + 8;                // fp32 staging pitch
constexpr int kWSmem = (int)(kWStages * 2 * kWOpBytes) > kWRows * kWStageLd * 4 ? (int)(kWStages * 2 * kWOpBytes)
                                                                                 : kWRows * kWStageLd * 4;

// Operand tile of a stage, both layouts 32 KB, 32-row (or 32-column) block x
// of the operand at byte 4096 x:
//  * k-major: 256 rows x 64 reduction values, 128 B per row, 16-byte chunk c
//    of row r at chunk c ^ ((r / 2) % 8), so each group of 16 lanes of a
//    fragment read (16 consecutive rows, one chunk) touches 16 distinct
//    16-byte bank groups;
//  * i-major: two plane tiles (tile_off) of 64 reduction rows x 128 columns,
//    columns 0..127 then 128..255, read with transposed 8-byte reads.
__device__ __forceinline__ uint32_t wide_off(int r, int c) { return (uint32_t)(r * 128 + ((c ^ ((r >> 1) & 7)) << 4)); }

// The direct loads of one wavefront: its share (pieces 8 sw .. 8 sw + 7 of
// the 32) of one operand's stage, the operand rows (k-major) or columns
// (i-major) r0 .. r0 + 255 of `src` (leading dimension ld, nrows of them).
// Piece q lands at dbase plus a per-piece constant (the kernel's issue):
// k-major pieces are 1 KB apart, i-major ones (plane-tile loads m = 8 (sw %
// 2) + q of column half sw / 2) q % 4 planes (4 KB) and q / 4 16-row groups
// (1 KB) from the wavefront's base.
struct WideLoad {
  uint32_t goff[kWPieces];
  uint32_t dbase;       // wavefront-uniform
  int64_t stage_bytes;  // global byte advance per stage
  const char* gbase;
  __device__ WideLoad(bool imajor, const bf16* src, int64_t ld, int64_t r0, int64_t nrows, int sw, int lane) {
#pragma unroll
    for (int q = 0; q < kWPieces; ++q) {
      const int P = kWPieces * sw + q;
      if (!imajor) {
        // rows 8 P .. 8 P + 7; lane l: row 8 P + l / 8, stored chunk l % 8
        const int r = 8 * P + (lane >> 3);
        const int c = (lane & 7) ^ ((r >> 1) & 7);
        const int64_t row = r0 + r < nrows ? r0 + r : nrows - 1;  // rows past the end re-read the last (never stored)
        goff[q] = (uint32_t)(((row - r0) * ld + 8 * c) * 2);
      } else {
        // plane-tile load m of column half P / 16
        const int half = P >> 4, m = P & 15;
        const int k = dma_row<kWBk>(m, lane);
        int64_t col = r0 + 128 * half + dma_col<kWBk>(m, lane);
        col = col < nrows ? col : nrows - 8;  // columns past the end re-read the last eight (never stored)
        goff[q] = (uint32_t)((k * ld + (col - r0)) * 2);
      }
    }
    dbase = imajor ? 16384u * (uint32_t)(sw >> 1) + 2048u * (uint32_t)(sw & 1) : 8192u * (uint32_t)sw;
    stage_bytes = imajor ? 2 * kWBk * ld : 2 * kWBk;
    gbase = reinterpret_cast<const char*>(src + (imajor ? r0 : r0 * ld));
  }
};

// Fragment reads of one operand: block x (32 rows or columns x 16
// reduction values, k-step ks; lane l holding row/column l % 32 and
// reduction values 16 ks + 8 (l / 32) + 0..7) is one 16-byte read
// (k-major) or two transposed reads of four reduction rows each (i-major).
template <bool kI>
struct WideFrag {
  uint32_t rd[kWKsteps];  // k-major: offset of block 0 per k-step
  uint32_t lo, hi;        // i-major: the two transposed-read offsets of block 0, k-step 0
  __device__ explicit WideFrag(int lane) {
    const int h = lane >> 5, i = lane & 15;
    if constexpr (!kI) {
#pragma unroll
      for (int ks = 0; ks < kWKsteps; ++ks) rd[ks] = wide_off(lane & 31, 2 * ks + h);
      lo = hi = 0;
    } else {
#pragma unroll
      for (int ks = 0; ks < kWKsteps; ++ks) rd[ks] = 0;
      lo = 2u * (uint32_t)tile_off<kWBk>(8 * h + (i >> 2), (lane & 16) + 4 * (i & 3));
      hi = 2u * (uint32_t)tile_off<kWBk>(8 * h + 4 + (i >> 2), (lane & 16) + 4 * (i & 3));
    }
  }
  template <int kKs>
  __device__ __forceinline__ bf16x8 frag(uint32_t T, uint32_t x) const {
    if constexpr (!kI) {
      return lds_ld16(T + 4096u * x + rd[kKs]);
    } else {
      const uint32_t c = T + 4096u * x + 1024u * kKs;
      const bf16x4 a = lds_ld_tr4(c + lo), b = lds_ld_tr4(c + hi);
      return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
    }
  }
};

}  // namespace

// One 256 x 256 output tile (index `tile`, row-major over the output's
// tiles) of the product in p, by the eight wavefronts of the workgroup.
// fr: the lane's eight rotary frequencies (q / k / v epilogue only)
template <bool kAI, bool kBI, int kEpi>
__device__ __forceinline__ void wide_tile(const ProjGemmParams& p, int64_t tile, unsigned char* smem_raw,
                                          const RopeFreq (&fr)[8]) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const int tiles_j = (p.J + kWTile - 1) / kWTile;
  const int64_t ti = tile / tiles_j;
  const int tj = (int)(tile - ti * tiles_j);
  const int64_t i0 = ti * kWTile;
  const int j0 = tj * kWTile;
  const int64_t nk = p.K / kWBk;

  // wavefronts 0-3 load A (rows / columns i0..), 4-7 B (j0..)
  const bool side_b = wave >= 4;
  const WideLoad ld = side_b ? WideLoad(kBI, p.b, p.ldb, j0, p.J, wave & 3, lane)
                             : WideLoad(kAI, p.a, p.lda, i0, p.I, wave & 3, lane);
  const uint32_t side_off = side_b ? kWOpBytes : 0u;
  const WideFrag<kAI> opa(lane);
  const WideFrag<kBI> opb(lane);
  const uint32_t lds0 = lds_addr(smem_raw);
  auto buf = [&](int64_t kt) { return lds0 + ((uint32_t)kt % kWStages) * 2u * kWOpBytes; };
  auto issue = [&](int64_t kt) {
    const int64_t ks = kt < nk ? kt : nk - 1;  // past the end: the last stage again, into its idle buffer
    const void* g = uniform_ptr(ld.gbase + ks * ld.stage_bytes);
    const uint32_t d = buf(kt) + side_off + ld.dbase;
#pragma unroll
    for (int q = 0; q < kWPieces; ++q) {
      const uint32_t ck = 1024u * q, ci = 4096u * (q & 3) + 1024u * (q >> 2);
      bool im;
      if constexpr (kAI == kBI) im = kAI;
      else im = side_b ? kBI : kAI;
      dma16_async(g, ld.goff[q], d + (im ? ci : ck));
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  // Fragments are read one k-step (16 reduction values) ahead, into the
  // other of two register sets, between the MFMAs of the current k-step.
  // The barrier that publishes stage kt+1 sits before the last k-step of
  // stage kt, whose reads (those of kt+1's first k-step) follow it; by then
  // every read of stage kt is done, so the loads of stage kt + 2 go into its
  // buffer right after that barrier.
  typedef bf16x8 Frags[6];  // A blocks 0..3, B blocks 0..1 of one k-step
  const uint32_t xa = 4u * wm, xb = 2u * wn;
  auto read = [&](uint32_t T, auto kc, int f) -> bf16x8 {
    constexpr int ks = decltype(kc)::value;
    return f < 4 ? opa.template frag<ks>(T, xa + f) : opb.template frag<ks>(T + kWOpBytes, xb + (f - 4));
  };
  // the eight MFMAs of a k-step from f, the six reads of the next one
  // (stage buffer T, k-step ks) into g between them (after the last k-step
  // they read an idle buffer, in bounds, and are not used)
  auto kstep = [&](const Frags& f, uint32_t T, auto kc, Frags& g) {
    static_for<8>([&](auto mc) {
      constexpr int m = decltype(mc)::value;
      constexpr int i = m >> 1, j = m & 1;
      acc[i][j] = mfma32(f[i], f[4 + j], acc[i][j]);
      if constexpr (m < 6) g[m] = read(T, kc, m);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  Frags f0, f1;
  if (nk > 0) {  // (an empty reduction loads nothing: the stage clamp needs one stage)
#pragma unroll
    for (int s0 = 0; s0 < kWStages; ++s0) issue(s0);
    wait_vmcnt_lgkm0<kWPieces * (kWStages - 1)>();  // stage 0 has landed for this wavefront
    lds_barrier();
#pragma unroll
    for (int m = 0; m < 6; ++m) f0[m] = read(buf(0), std::integral_constant<int, 0>{}, m);
  }
  for (int64_t kt = 0; kt < nk; ++kt) {
    const uint32_t T = buf(kt);
    kstep(f0, T, std::integral_constant<int, 1>{}, f1);
    kstep(f1, T, std::integral_constant<int, 2>{}, f0);
    kstep(f0, T, std::integral_constant<int, 3>{}, f1);
    wait_vmcnt_lgkm0<kWPieces * (kWStages - 2)>();  // stage kt+1 has landed
    lds_barrier();
    issue(kt + kWStages);  // into stage kt's buffer, read completely before the barrier
    kstep(f1, buf(kt + 1), std::integral_constant<int, 0>{}, f0);  // the last k-step; reads of stage kt+1's first
  }
  __builtin_amdgcn_s_waitcnt(0);  // no direct load outlives the loop
  __syncthreads();

  // accumulator element v of lane l: row 8 (v/4) + 4 (l/32) + v%4, column l%32
  if constexpr (kEpi == kProjEpiPlain) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int64_t col = j0 + 64 * wn + 32 * j + (lane & 31);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int64_t row = i0 + 128 * wm + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
          if (row < p.I && col < p.J) {
            const int64_t at = row * p.ldc + col;
            if (p.c_f32) {
              float* c = static_cast<float*>(p.c);
              c[at] = p.accumulate ? c[at] + acc[i][j][v] : acc[i][j][v];
            } else {
              static_cast<bf16*>(p.c)[at] = (bf16)acc[i][j][v];
            }
          }
        }
      }
    return;
  }

  // ---- epilogue: two passes of 128 rows staged in fp32 (the wavefronts of
  // row half wm write in pass wm), then one 16-lane row per output row and
  // both heads of the tile: lane l16 holds dims 8 l16 .. +7 of each, its
  // rotation partner (dims +-64) in lane l16 ^ 8 of the same DPP row.  Accumulator element v of lane l:
  // row 8 (v/4) + 4 (l/32) + v%4, column l%32.
  float* S = reinterpret_cast<float*>(smem_raw);
  const int l16 = tid & 15;
  const float sg = l16 < 8 ? -1.f : 1.f;
  const int heads = p.J / kHeadDim;

  for (int pass = 0; pass < 2; ++pass) {
    if (wm == pass) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            S[(32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * kWStageLd + 64 * wn + 32 * j + (lane & 31)] =
                acc[i][j][v];
    }
    __syncthreads();
    // one row of both heads per task, the angles of a row once for both
    for (int rr = 0; rr < kWRows / 32; ++rr) {
      const int r = (tid >> 4) + 32 * rr;
      const int64_t row = i0 + kWRows * pass + r;
      bf16* dst[2];
      int hh[2], nh[2];
      bool live[2], rot[2];
#pragma unroll
      for (int hs = 0; hs < 2; ++hs) {
        const int head = 2 * tj + hs;
        live[hs] = head < heads && row < p.I;
        if (head < p.hq) {
          dst[hs] = p.q; hh[hs] = head; nh[hs] = p.hq;
        } else if (head < p.hq + p.hkv) {
          dst[hs] = p.k; hh[hs] = head - p.hq; nh[hs] = p.hkv;
        } else {
          dst[hs] = p.v; hh[hs] = head - p.hq - p.hkv; nh[hs] = p.hkv;
        }
        rot[hs] = p.rotate && head < p.hq + p.hkv;
      }
      float x[2][8];
#pragma unroll
      for (int hs = 0; hs < 2; ++hs) {
        const float* sr = S + r * kWStageLd + kHeadDim * hs + 8 * l16;
        const float4 x0 = *reinterpret_cast<const float4*>(sr);
        const float4 x1 = *reinterpret_cast<const float4*>(sr + 4);
        x[hs][0] = x0.x; x[hs][1] = x0.y; x[hs][2] = x0.z; x[hs][3] = x0.w;
        x[hs][4] = x1.x; x[hs][5] = x1.y; x[hs][6] = x1.z; x[hs][7] = x1.w;
      }
      const int ps = ((rot[0] || rot[1]) && row < p.I) ? p.pos[row] : -1;
      float y[2][8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float sn = 0.f, cs = 1.f;
        if (ps >= 0) rope_sincos_fast(ps, fr[e], sn, cs);
#pragma unroll
        for (int hs = 0; hs < 2; ++hs) {
          const float xp = dpp_mov<0x128>(x[hs][e]);  // row_ror:8, the partner lane l16 ^ 8
          y[hs][e] = rot[hs] ? fmaf(xp, sn * sg, x[hs][e] * cs) : x[hs][e];
        }
      }
#pragma unroll
      for (int hs = 0; hs < 2; ++hs)
        if (live[hs])
          st16(dst[hs] + (row * nh[hs] + hh[hs]) * kHeadDim + 8 * l16,
               pack8(y[hs][0], y[hs][1], y[hs][2], y[hs][3], y[hs][4], y[hs][5], y[hs][6], y[hs][7]));
    }
    __syncthreads();
  }
}

template <bool kAI, bool kBI, int kEpi>
__global__ __launch_bounds__(512, 1) void proj_gemm_wide_kernel(const ProjGemmParams p) {
  __shared__ __align__(16) unsigned char smem_raw[kWSmem];
  // the lane's frequencies (dim pairs 8 (l % 8) + e of lane l of a 16-lane
  // row), picked with compile-time indices: with the parameter block also
  // passed by reference, a run-time index into it makes the compiler keep a
  // copy of the whole block in scratch memory
  RopeFreq fr[8];
  if constexpr (kEpi == kProjEpiQkv) {
    const int fsel = threadIdx.x & 7;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      RopeFreq v = p.freq.f[e];
#pragma unroll
      for (int k = 1; k < 8; ++k)
        if (fsel == k) v = p.freq.f[8 * k + e];
      fr[e] = v;
    }
  }
  wide_tile<kAI, kBI, kEpi>(p, blockIdx.x, smem_raw, fr);
}

// The backward's two products in one launch: the tiles of dW = dY^T X (pw,
// both operands i-major, a reduction over all rows) first, then those of dX
// = dY W (px).  dW has few, long tiles (384 at hidden 4096 and 48 heads, a
// round and a half on 256 compute units); dX's many short ones then fill
// the compute units that dW's last round leaves idle.
__global__ __launch_bounds__(512, 1) void proj_gemm_wide_bwd_kernel(const ProjGemmParams pw, const ProjGemmParams px,
                                                                    int64_t tiles_w) {
  __shared__ __align__(16) unsigned char smem_raw[kWSmem];
  const RopeFreq none[8] = {};
  if ((int64_t)blockIdx.x < tiles_w) wide_tile<true, true, kProjEpiPlain>(pw, blockIdx.x, smem_raw, none);
  else wide_tile<false, true, kProjEpiPlain>(px, (int64_t)blockIdx.x - tiles_w, smem_raw, none);
}

namespace {

__device__ __forceinline__ void load8f(const bf16* p, float (&x)[8]) {
  const bf16x8 v = ld16(p);
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = (float)v[e];
}
__device__ __forceinline__ void load8f(const float* p, float (&x)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

constexpr int kPackHeads = 4;  // heads loaded together, before any is used

}  // namespace

// dY[row] = [R(pos)^T dq[row], R(pos)^T dk[row], dv[row]] in bf16, one
// 16-lane DPP row per token row (rows with a negative position, or every row
// when rotate == 0, are copied unrotated).
template <typename Src>
__global__ __launch_bounds__(256) void proj_grad_pack_kernel(const Src* __restrict__ dq, const Src* __restrict__ dk,
                                                             const Src* __restrict__ dv, bf16* __restrict__ dy,
                                                             const int32_t* __restrict__ pos, int64_t rows, int hq,
                                                             int hkv, int rotate, const RopeFreqTable freq) {
  const int lane = threadIdx.x & 63;
  const int64_t r0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
  const int64_t r = r0 < rows ? r0 : rows - 1;  // rows past the end redo the last row and write nothing
  const bool live = r0 < rows;
  const int ps = rotate ? pos[r] : -1;
  const int l = lane & 15;
  const float sg = l < 8 ? 1.f : -1.f;
  float cs[8], sn[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    cs[e] = 1.f;
    sn[e] = 0.f;
  }
  if (ps >= 0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      rope_sincos(ps, freq.f[8 * (l & 7) + e], sn[e], cs[e]);
      sn[e] *= sg;
    }
  }
  const int heads = hq + 2 * hkv;
  bf16* out = dy + r * (int64_t)heads * kHeadDim + 8 * l;
  for (int h0 = 0; h0 < heads; h0 += kPackHeads) {
    float x[kPackHeads][8];
#pragma unroll
    for (int u = 0; u < kPackHeads; ++u) {
      const int h = h0 + u < heads ? h0 + u : h0;
      const Src* src = h < hq ? dq + (r * hq + h) * kHeadDim
                              : (h < hq + hkv ? dk + (r * hkv + (h - hq)) * kHeadDim
                                              : dv + (r * hkv + (h - hq - hkv)) * kHeadDim);
      load8f(src + 8 * l, x[u]);
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the loads together, ahead of their uses
#pragma unroll
    for (int u = 0; u < kPackHeads; ++u) {
      const int h = h0 + u;
      const bool turn = h < hq + hkv;
      float y[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xp = dpp_mov<0x128>(x[u][e]);  // row_ror:8, the partner lane l ^ 8
        y[e] = turn ? fmaf(xp, sn[e], x[u][e] * cs[e]) : x[u][e];
      }
      if (live && h < heads) st16(out + (int64_t)h * kHeadDim, pack8(y[0], y[1], y[2], y[3], y[4], y[5], y[6], y[7]));
    }
  }
}

hipError_t launch_proj_gemm(const ProjGemmParams& p, bool a_imajor, bool b_imajor, int epi, hipStream_t stream) {
  const int64_t tiles = ((p.I + kTile - 1) / kTile) * (p.J / kTile);
  if (tiles <= 0) return hipSuccess;
  const dim3 grid((unsigned)tiles), block(256);
  if (proj_gemm_wide_ok(p)) {
    const dim3 wgrid((unsigned)(((p.I + kWTile - 1) / kWTile) * ((p.J + kWTile - 1) / kWTile))), wblock(512);
    if (epi == kProjEpiQkv && !a_imajor && !b_imajor)
      hipLaunchKernelGGL((proj_gemm_wide_kernel<false, false, kProjEpiQkv>), wgrid, wblock, 0, stream, p);
    else if (epi == kProjEpiPlain && !a_imajor && b_imajor)
      hipLaunchKernelGGL((proj_gemm_wide_kernel<false, true, kProjEpiPlain>), wgrid, wblock, 0, stream, p);
    else if (epi == kProjEpiPlain && a_imajor && b_imajor)
      hipLaunchKernelGGL((proj_gemm_wide_kernel<true, true, kProjEpiPlain>), wgrid, wblock, 0, stream, p);
    else
      return hipErrorInvalidValue;
  } else if (epi == kProjEpiQkv && !a_imajor && !b_imajor)
    hipLaunchKernelGGL((proj_gemm_kernel<false, false, kProjEpiQkv>), grid, block, 0, stream, p);
  else if (epi == kProjEpiPlain && !a_imajor && b_imajor)
    hipLaunchKernelGGL((proj_gemm_kernel<false, true, kProjEpiPlain>), grid, block, 0, stream, p);
  else if (epi == kProjEpiPlain && a_imajor && b_imajor)
    hipLaunchKernelGGL((proj_gemm_kernel<true, true, kProjEpiPlain>), grid, block, 0, stream, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

bool proj_gemm_wide_ok(const ProjGemmParams& p) { return p.K > 0 && p.K % kWBk == 0; }

hipError_t launch_proj_gemm_bwd_pair(const ProjGemmParams& pw, const ProjGemmParams& px, hipStream_t stream) {
  const int64_t tw = ((pw.I + kWTile - 1) / kWTile) * ((pw.J + kWTile - 1) / kWTile);
  const int64_t tx = ((px.I + kWTile - 1) / kWTile) * ((px.J + kWTile - 1) / kWTile);
  if (tw + tx <= 0) return hipSuccess;
  hipLaunchKernelGGL(proj_gemm_wide_bwd_kernel, dim3((unsigned)(tw + tx)), dim3(512), 0, stream, pw, px, tw);
  return hipGetLastError();
}

hipError_t launch_proj_grad_pack(const void* dq, const void* dk, const void* dv, bool src_f32, bf16* dy,
                                 const int32_t* pos, int64_t rows, int hq, int hkv, bool rotate,
                                 const RopeFreqTable& freq, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows * 16 + 255) / 256)), block(256);
  if (src_f32)
    hipLaunchKernelGGL((proj_grad_pack_kernel<float>), grid, block, 0, stream, static_cast<const float*>(dq),
                       static_cast<const float*>(dk), static_cast<const float*>(dv), dy, pos, rows, hq, hkv,
                       rotate ? 1 : 0, freq);
  else
    hipLaunchKernelGGL((proj_grad_pack_kernel<bf16>), grid, block, 0, stream, static_cast<const bf16*>(dq),
                       static_cast<const bf16*>(dk), static_cast<const bf16*>(dv), dy, pos, rows, hq, hkv,
                       rotate ? 1 : 0, freq);
  return hipGetLastError();
}

}  // namespace ba

// ------------------------------------------------------------------ C ABI

namespace {

int proj_fail(int code, const std::string& msg) {
  ba::set_error(msg);
  return code;
}

bool misaligned(const void* p) { return ((uintptr_t)p & 15) != 0; }

// shared argument checks of the forward and backward calls
int proj_check(int64_t rows, int32_t hidden, int32_t hq, int32_t hkv, const void* x, const void* w,
               const int32_t* pos, float theta) {
  if (rows < 0) return proj_fail(BA_E_INVAL, "qkv: rows must be >= 0");
  if (hidden <= 0 || hidden % 128 != 0) return proj_fail(BA_E_UNSUPPORTED, "qkv: hidden must be a positive multiple of 128");
  if (hq < 1 || hkv < 1 || hq % hkv != 0) return proj_fail(BA_E_INVAL, "qkv: need hq >= 1, hkv >= 1 and hq % hkv == 0");
  if (!std::isfinite(theta) || theta < 0.f) return proj_fail(BA_E_INVAL, "qkv: theta must be finite and >= 0");
  if ((int64_t)(hq + 2 * hkv) * ((rows + 127) / 128) > 0x7fffffffLL)
    return proj_fail(BA_E_UNSUPPORTED, "qkv: too many output tiles for one launch");
  if (rows > 0) {
    if (!x || !w) return proj_fail(BA_E_INVAL, "qkv: x or w is NULL");
    if (misaligned(x) || misaligned(w)) return proj_fail(BA_E_INVAL, "qkv: x and w must be 16-byte aligned");
    if (theta > 0.f && !pos) return proj_fail(BA_E_INVAL, "qkv: pos is NULL with theta > 0");
  }
  return BA_OK;
}

ba::RopeFreqTable freq_table(float theta) {
  ba::RopeFreqTable t{};
  if (theta > 0.f) ba::rope_freq_table(theta, t.f);
  return t;
}

}  // namespace

extern "C" int branch_attn_qkv_workspace_size(int64_t rows, int32_t hq, int32_t hkv, size_t* bytes) {
  if (rows < 0 || hq < 1 || hkv < 1) return proj_fail(BA_E_INVAL, "qkv workspace: need rows >= 0, hq >= 1, hkv >= 1");
  if (!bytes) return proj_fail(BA_E_INVAL, "qkv workspace: bytes is NULL");
  *bytes = (size_t)rows * (size_t)(hq + 2 * hkv) * ba::kHeadDim * sizeof(uint16_t);
  return BA_OK;
}

extern "C" int branch_attn_qkv_fwd(void* stream, int64_t rows, int32_t hidden, int32_t hq, int32_t hkv,
                                   const void* x, const void* w, const int32_t* pos, float theta, void* q,
                                   void* k, void* v) {
  int rc = proj_check(rows, hidden, hq, hkv, x, w, pos, theta);
  if (rc) return rc;
  if (rows == 0) return BA_OK;
  if (!q || !k || !v) return proj_fail(BA_E_INVAL, "qkv: q, k or v is NULL");
  if (misaligned(q) || misaligned(k) || misaligned(v)) return proj_fail(BA_E_INVAL, "qkv: q, k and v must be 16-byte aligned");
  ba::ProjGemmParams p{};
  p.a = static_cast<const ba::bf16*>(x);
  p.b = static_cast<const ba::bf16*>(w);
  p.lda = hidden;
  p.ldb = hidden;
  p.I = rows;
  p.J = (hq + 2 * hkv) * ba::kHeadDim;
  p.K = hidden;
  p.q = static_cast<ba::bf16*>(q);
  p.k = static_cast<ba::bf16*>(k);
  p.v = static_cast<ba::bf16*>(v);
  p.hq = hq;
  p.hkv = hkv;
  p.rotate = theta > 0.f ? 1 : 0;
  p.pos = pos;
  p.freq = freq_table(theta);
  const hipError_t e = ba::launch_proj_gemm(p, false, false, ba::kProjEpiQkv, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return proj_fail(BA_E_HIP, std::string("qkv forward launch: ") + hipGetErrorString(e));
  return BA_OK;
}

extern "C" int branch_attn_qkv_bwd(void* stream, int64_t rows, int32_t hidden, int32_t hq, int32_t hkv,
                                   const void* x, const void* w, const int32_t* pos, float theta, const void* dq,
                                   const void* dk, const void* dv, int32_t grad_dtype, void* dx, int32_t dx_dtype,
                                   float* dw, int32_t accumulate_dw, void* workspace, size_t workspace_bytes) {
  int rc = proj_check(rows, hidden, hq, hkv, x, w, pos, theta);
  if (rc) return rc;
  if (grad_dtype != BA_DTYPE_BF16 && grad_dtype != BA_DTYPE_F32)
    return proj_fail(BA_E_INVAL, "qkv: grad_dtype must be BA_DTYPE_BF16 or BA_DTYPE_F32");
  if (dx_dtype != BA_DTYPE_BF16 && dx_dtype != BA_DTYPE_F32)
    return proj_fail(BA_E_INVAL, "qkv: dx_dtype must be BA_DTYPE_BF16 or BA_DTYPE_F32");
  if (!dw || misaligned(dw)) return proj_fail(BA_E_INVAL, "qkv: dw is NULL or not 16-byte aligned");
  if (rows > 0) {
    if (!dq || !dk || !dv || !dx) return proj_fail(BA_E_INVAL, "qkv: dq, dk, dv or dx is NULL");
    if (misaligned(dq) || misaligned(dk) || misaligned(dv) || misaligned(dx))
      return proj_fail(BA_E_INVAL, "qkv: dq, dk, dv and dx must be 16-byte aligned");
  }
  size_t need = 0;
  branch_attn_qkv_workspace_size(rows, hq, hkv, &need);
  if (rows > 0 && (!workspace || workspace_bytes < need))
    return proj_fail(BA_E_WORKSPACE, "qkv: workspace of " + std::to_string(workspace_bytes) + " bytes, need " +
                                         std::to_string(need));
  if (rows > 0 && ((uintptr_t)workspace & 255)) return proj_fail(BA_E_WORKSPACE, "qkv: workspace must be 256-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int32_t n = (hq + 2 * hkv) * ba::kHeadDim;
  ba::bf16* dy = static_cast<ba::bf16*>(workspace);
  const ba::RopeFreqTable ft = freq_table(theta);
  hipError_t e = ba::launch_proj_grad_pack(dq, dk, dv, grad_dtype == BA_DTYPE_F32, dy, pos, rows, hq, hkv, theta > 0.f,
                                           ft, s);
  if (e != hipSuccess) return proj_fail(BA_E_HIP, std::string("qkv gradient pack launch: ") + hipGetErrorString(e));
  // dX [rows, hidden] = dY [rows, n] W [n, hidden]: A k-major, B i-major
  ba::ProjGemmParams px{};
  px.a = dy;
  px.lda = n;
  px.b = static_cast<const ba::bf16*>(w);
  px.ldb = hidden;
  px.I = rows;
  px.J = hidden;
  px.K = n;
  px.c = dx;
  px.ldc = hidden;
  px.c_f32 = dx_dtype == BA_DTYPE_F32;
  px.accumulate = 0;
  // dW [n, hidden] (+)= dY^T X: A = dY read i-major, B = X read i-major,
  // reduction over the rows (ragged end allowed)
  ba::ProjGemmParams pw{};
  pw.a = dy;
  pw.lda = n;
  pw.b = static_cast<const ba::bf16*>(x);
  pw.ldb = hidden;
  pw.I = n;
  pw.J = hidden;
  pw.K = rows;
  pw.c = dw;
  pw.ldc = hidden;
  pw.c_f32 = 1;
  pw.accumulate = accumulate_dw ? 1 : 0;
  if (ba::proj_gemm_wide_ok(px) && ba::proj_gemm_wide_ok(pw)) {
    if ((e = ba::launch_proj_gemm_bwd_pair(pw, px, s)) != hipSuccess)
      return proj_fail(BA_E_HIP, std::string("qkv dW + dX launch: ") + hipGetErrorString(e));
    return BA_OK;
  }
  if ((e = ba::launch_proj_gemm(px, false, true, ba::kProjEpiPlain, s)) != hipSuccess)
    return proj_fail(BA_E_HIP, std::string("qkv dX launch: ") + hipGetErrorString(e));
  if ((e = ba::launch_proj_gemm(pw, true, true, ba::kProjEpiPlain, s)) != hipSuccess)
    return proj_fail(BA_E_HIP, std::string("qkv dW launch: ") + hipGetErrorString(e));
  return BA_OK;
}
