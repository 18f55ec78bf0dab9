// Internal data structures shared by the host planner and the gfx950 kernels.
//
// The planner turns a rank share (Sec. 3.2 of the paper: main queries of the
// rank's two zigzag chunks, branch groups anchored there) into flat tables
// that the kernels index directly:
//   * SeqInfo   -- per sequence: where its keys sit in every ring-step block
//                  and which slice of the token table holds its queries;
//   * TokInfo   -- per query token, ordered by causal limit P within a
//                  sequence (main token at p has P = p; a branch member has
//                  P = anchor), so that every key tile is read by a
//                  contiguous range of tokens;
//   * GroupInfo -- per branch group: member rows and kind;
//   * FwdTile   -- a forward work item: up to kFwdRows / G tokens times the G
//                  query heads of one KV head;
//   * BwdTile   -- a backward work item: kBwdKeys keys of one ring-step
//                  block, one sequence and one KV head, plus the range of
//                  query tokens that reach them.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "branch_attn.h"

namespace ba {

// tile shapes (the kernels are written for exactly these)
constexpr int kHeadDim = 128;
constexpr int kFwdRows = 256;   // query rows (token x head) per forward tile
constexpr int kFwdKeys = 64;    // keys per forward inner iteration
constexpr int kBwdKeys = 128;   // keys owned by one backward work item
constexpr int kBwdRows = 64;    // query rows per backward inner iteration

struct SeqInfo {
  int32_t seg_off;    // offset of the sequence in every rank-local main array
  int32_t c;          // zigzag chunk length L / (2 C)
  int32_t tok_begin;  // query tokens of the sequence: [tok_begin, tok_end)
  int32_t tok_end;
};

struct TokInfo {
  int32_t qrow;  // >= 0: rank-local main row; < 0: branch row (-qrow - 1)
  int32_t P;     // causal limit: keys at positions 0..P are visible
  int32_t grp;   // branch group, -1 for a main token
  int32_t gidx;  // member index inside the group
};

struct GroupInfo {
  int32_t row0;
  int32_t stride;
  int32_t len;
  int32_t kind;
  int32_t tok0;  // token-table index of member 0 (members are consecutive)
  int32_t anchor;
  int32_t pad[2];
};

// Rotary embedding frequency of dim pair j: theta^(-j/64) / (2 pi) turns per
// position, as an unevaluated float sum hi + lo.
struct RopeFreq {
  float hi, lo;
};

// The 64 frequencies of base theta (> 0), computed in double and split.
void rope_freq_table(float theta, RopeFreq* out);
// The same 64 frequencies in radians per position, theta^(-j/64), in double:
// the rotation of the attention's inputs takes its angles, sine, cosine and
// products in double and rounds once to bf16.
void rope_rad_table(float theta, double* out);

// sin and cos of the angle of dim pair f at position pos.  The turns
// pos * f are formed as an unevaluated float sum, the product's rounding
// error recovered with an fma, and the whole turns are removed before the
// sum is rounded, so the angle stays within ~1e-7 rad of the exact one at
// every position below 2^24.  Contraction stays off: fusing p * hi into
// the subtraction of the whole turns would count the product's rounding
// error twice (once there, once in tl), an angle error of up to half an ulp
// of the turn count.
__device__ __forceinline__ void rope_sincos(int pos, RopeFreq f, float& s, float& c) {
#pragma clang fp contract(off)
  const float p = (float)pos;
  const float th = p * f.hi;
  const float tl = fmaf(p, f.lo, fmaf(p, f.hi, -th));
  const float r = (th - rintf(th)) + tl;  // fraction of a turn in [-0.5, 0.5]
  sincospif(2.f * r, &s, &c);
}
// The same angle reduction, then the hardware sine and cosine, which take
// their argument in turns (v_sin_f32 / v_cos_f32: a few instructions instead
// of a library evaluation; over turn fractions in [-0.5, 0.5] their
// absolute error measured at most 1.3e-7).
__device__ __forceinline__ void rope_sincos_fast(int pos, RopeFreq f, float& s, float& c) {
#pragma clang fp contract(off)
  const float p = (float)pos;
  const float th = p * f.hi;
  const float tl = fmaf(p, f.lo, fmaf(p, f.hi, -th));
  const float r = (th - rintf(th)) + tl;
  s = __builtin_amdgcn_sinf(r);
  c = __builtin_amdgcn_cosf(r);
}

struct FwdTile {
  int32_t seq;
  int32_t tok_begin;
  int32_t ntok;
  int32_t kvh;
  // branch-local keys of the tile's tokens: rows br_keys[bk_off ..
  // bk_off + bk_n) of the branch K/V arrays, each group's keys consecutive
  // (a token's group starts at its tok_bslot); bk_n = -1: more than
  // kBrSlots keys, the rows read their keys from global memory instead
  int32_t bk_off;
  int32_t bk_n;
};

// LDS staging of a forward tile's branch-local keys in the fused epilogue:
// K rows then V rows of up to kBrSlots keys, kBrPitch bytes apart (256 bytes
// of data plus 16 of padding, so rows of different keys start in different
// bank groups)
constexpr int32_t kBrSlots = 288;
constexpr int32_t kBrPitch = 272;

struct BwdTile {
  int32_t step;     // ring step block j
  int32_t seq;
  int32_t kvh;
  int32_t u0;       // first key, as an index inside the sequence's segment
  int32_t nk;       // keys in this item (<= kBwdKeys)
  int32_t q_begin;  // first token of the item that sees at least one of the keys
  int32_t q_full;   // tokens >= q_full see all of them
  int32_t q_end;
  int32_t slot;     // -1: the item writes dK, dV; else its fp32 partial slot
  int32_t walk_down;  // 1: query tiles from the last down, 0: from the first up
  int32_t pad[2];
};

// Keys whose query range was split into several work items: the items'
// fp32 partial dK, dV (slots slot0 .. slot0 + nslots - 1) are summed into
// the outputs afterwards.
struct KvSplit {
  int32_t step;
  int32_t key0;  // first key row in block `step` (segment offset + u0)
  int32_t kvh;
  int32_t nk;
  int32_t slot0;
  int32_t nslots;
  int32_t pad[2];
};

// A ring step whose backward work items number fewer than this has its
// longest items split along the query range, so one launch still fills the
// GPU (four items per compute unit of an MI355X).
constexpr int32_t kKvSplitBelow = 1024;
// dK/dV work items that start together on the GPU: one per compute unit
// (MI355X: 256), one workgroup per compute unit.  Only the items' walk
// direction depends on it (an L2 locality choice, no effect on results).
constexpr int32_t kKvRoundItems = 256;
// smallest piece of a split item, in 64-row query tiles
constexpr int32_t kKvSplitMinTiles = 16;

// Number of keys of ring-step block j (rank j's chunks j and 2C-1-j of a
// sequence with chunk length c) at positions <= P.  Positions increase with
// the local index inside the block, so the visible keys are a prefix.
__host__ __device__ inline int32_t visible_keys(int32_t P, int32_t j, int32_t C, int32_t c) {
  int32_t a = P - j * c + 1;
  int32_t b = P - (2 * C - 1 - j) * c + 1;
  a = a < 0 ? 0 : (a > c ? c : a);
  b = b < 0 ? 0 : (b > c ? c : b);
  return a + b;
}

struct Plan {
  // problem
  int32_t num_seqs = 0, cp_size = 1, cp_rank = 0, hq = 0, hkv = 0, head_dim = 0, group = 1;
  float scale = 0.f;
  int64_t n_local = 0;
  int32_t num_branch_rows = 0;
  bool any_main_query = false;
  std::vector<int32_t> cu_seqlens;
  // tables (host copies, uploaded into the workspace per call)
  std::vector<SeqInfo> seqs;
  std::vector<TokInfo> toks;
  std::vector<GroupInfo> groups;
  std::vector<FwdTile> fwd_tiles;
  std::vector<int32_t> br_keys;        // branch key rows of the forward tiles (see FwdTile)
  std::vector<int32_t> tok_bslot;      // per token: first slot of its group's keys in its tile, -1 main
  std::vector<BwdTile> bwd_tiles;      // grouped by ring step i = 0..C-1
  std::vector<int32_t> bwd_step_off;   // [C+1] tile range of each ring step
  std::vector<KvSplit> kv_splits;      // keys whose items write partial sums
  int32_t kv_slots = 0;                // partial slots in use
  // packed image of the tables and their byte offsets inside it
  std::vector<uint8_t> image;
  size_t off_seqs = 0, off_toks = 0, off_groups = 0, off_fwd = 0, off_bwd = 0, off_splits = 0;
  size_t off_br_keys = 0, off_bslot = 0;
  // rotary position embedding (off while rope_theta == 0): positions of the
  // rows of every ring-step block ([C][n_local], block j = rank j's local
  // rows), of this rank's main rows that are queries and of the branch rows
  // in a group (-1 elsewhere: such rows are neither read nor written), and
  // the frequency table
  float rope_theta = 0.f;
  std::vector<int32_t> pos_block;
  std::vector<int32_t> pos_qmain;
  std::vector<int32_t> pos_br;
  std::vector<RopeFreq> rope_freq;
  std::vector<double> rope_rad;
  size_t off_pos_block = 0, off_pos_qmain = 0, off_pos_br = 0, off_freq = 0, off_rad = 0;
  // counts
  double pairs_per_head = 0.0;  // allowed (query, key) pairs per query head
  double main_pairs_per_head = 0.0;   // ... of which on the causal main prefix
  int32_t max_group_len = 0;
  // schedule BA_MODE_AUTO resolves to (fused; see build_plan)
  int32_t auto_mode = 1;
};

// BA_MODE_AUTO -> the plan's choice; other values unchanged
inline int32_t resolve_mode(const Plan& p, int32_t mode) { return mode == BA_MODE_AUTO ? p.auto_mode : mode; }

// workspace layout (byte offsets), computed from a plan
struct WorkspaceLayout {
  size_t tables = 0;   // start of the table image
  size_t o_acc = 0;    // fp32 [T, hq, d]   (per-step forward)
  size_t lse_acc = 0;  // fp32 [T, hq]      (per-step forward)
  size_t rowstat = 0;  // float2 [T, hq]    (backward: -LSE*log2e, -Delta)
  size_t qtok = 0;     // bf16 [T, hq, d]   (backward: Q in token order)
  size_t gtok = 0;     // bf16 [T, hq, d]   (backward: dO in token order)
  size_t dq_acc = 0;   // fp32 [T, hq, d]   (backward)
  size_t kv_part = 0;  // fp32 [slots][dV, dK][kBwdKeys][d] (backward, split items)
  // rotary embedding: rotated bf16 copies of the inputs (both passes) and
  // fp32 staging of the gradients (backward)
  size_t rq_main = 0, rq_br = 0, rk_step = 0, rk_br = 0;
  size_t gq_main = 0, gq_br = 0, gk_step = 0, gv_step = 0, gk_br = 0, gv_br = 0;
  size_t fwd_total = 0;
  size_t bwd_total = 0;
};

WorkspaceLayout workspace_layout(const Plan& p, int mode);

// (re)build the packed table image of a plan
void pack_image(Plan& P);

// thread-local error message
void set_error(const std::string& msg);

}  // namespace ba

struct ba_plan {
  ba::Plan p;
};
