// Host planner: zigzag partition, descriptor validation and the work tables
// the kernels consume.  Host code only (no HIP runtime calls).
#include <algorithm>
#include <exception>
#include <new>
#include <cmath>
#include <cstring>
#include <numeric>
#include <string>
#include <vector>

#include "ba_internal.h"

namespace ba {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }

static int fail(int code, const std::string& msg) {
  set_error(msg);
  return code;
}

static int check_seqlens(const int32_t* cu, int32_t num_seqs, int32_t cp_size, int32_t cp_rank) {
  if (!cu) return fail(BA_E_INVAL, "cu_seqlens is NULL");
  if (num_seqs < 1) return fail(BA_E_INVAL, "num_seqs must be >= 1");
  if (cp_size < 1) return fail(BA_E_INVAL, "cp_size must be >= 1");
  if (cp_rank < 0 || cp_rank >= cp_size) return fail(BA_E_INVAL, "cp_rank outside [0, cp_size)");
  if (cu[0] != 0) return fail(BA_E_INVAL, "cu_seqlens[0] must be 0");
  for (int32_t s = 0; s < num_seqs; ++s) {
    int64_t L = (int64_t)cu[s + 1] - cu[s];
    if (L < 0) return fail(BA_E_INVAL, "cu_seqlens must be non-decreasing");
    if (L % (2 * (int64_t)cp_size) != 0)
      return fail(BA_E_INVAL, "sequence " + std::to_string(s) + " length " + std::to_string(L) +
                                  " is not a multiple of 2*cp_size");
  }
  return BA_OK;
}

WorkspaceLayout workspace_layout(const Plan& p, int mode) {
  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  WorkspaceLayout w;
  size_t T = p.toks.size();
  size_t rows = T * (size_t)p.hq;
  const bool rope = p.rope_theta > 0.f;
  const size_t nl = (size_t)p.n_local, nb = (size_t)p.num_branch_rows, C = (size_t)p.cp_size;
  const size_t qrow = (size_t)p.hq * kHeadDim, krow = (size_t)p.hkv * kHeadDim;
  size_t off = 0;
  w.tables = off;
  off = align(off + p.image.size());
  if (rope) {  // rotated inputs, shared by the forward and backward layouts
    w.rq_main = off;
    off = align(off + nl * qrow * sizeof(uint16_t));
    w.rq_br = off;
    off = align(off + nb * qrow * sizeof(uint16_t));
    w.rk_step = off;
    off = align(off + C * nl * krow * sizeof(uint16_t));
    w.rk_br = off;
    off = align(off + nb * krow * sizeof(uint16_t));
  }
  const size_t common = off;
  if (mode == BA_MODE_PER_STEP) {
    w.o_acc = off;
    off = align(off + rows * kHeadDim * sizeof(float));
    w.lse_acc = off;
    off = align(off + rows * sizeof(float));
  }
  w.fwd_total = off;
  off = common;
  w.rowstat = off;
  off = align(off + rows * 2 * sizeof(float));
  w.qtok = off;
  off = align(off + rows * kHeadDim * sizeof(uint16_t));
  w.gtok = off;
  off = align(off + rows * kHeadDim * sizeof(uint16_t));
  if (mode == BA_MODE_PER_STEP) {
    w.dq_acc = off;
    off = align(off + rows * kHeadDim * sizeof(float));
  }
  if (p.kv_slots > 0) {
    w.kv_part = off;
    off = align(off + (size_t)p.kv_slots * 2 * kBwdKeys * kHeadDim * sizeof(float));
  }
  if (rope) {
    w.gq_main = off;
    off = align(off + nl * qrow * sizeof(float));
    w.gq_br = off;
    off = align(off + nb * qrow * sizeof(float));
    w.gk_step = off;
    off = align(off + C * nl * krow * sizeof(float));
    w.gv_step = off;
    off = align(off + C * nl * krow * sizeof(float));
    w.gk_br = off;
    off = align(off + nb * krow * sizeof(float));
    w.gv_br = off;
    off = align(off + nb * krow * sizeof(float));
  }
  w.bwd_total = off;
  return w;
}

template <typename T>
static size_t append(std::vector<uint8_t>& img, const std::vector<T>& v) {
  size_t off = (img.size() + 255) & ~size_t(255);
  img.resize(off + v.size() * sizeof(T));
  if (!v.empty()) std::memcpy(img.data() + off, v.data(), v.size() * sizeof(T));
  return off;
}

static int build_plan(const ba_problem* pr, Plan& P) {
  int rc = check_seqlens(pr->cu_seqlens, pr->num_seqs, pr->cp_size, pr->cp_rank);
  if (rc) return rc;
  if (pr->head_dim != kHeadDim)
    return fail(BA_E_UNSUPPORTED, "head_dim " + std::to_string(pr->head_dim) + " unsupported (only 128)");
  if (pr->hq < 1 || pr->hkv < 1 || pr->hq % pr->hkv != 0)
    return fail(BA_E_INVAL, "hq and hkv must be positive with hq % hkv == 0");
  const int32_t G = pr->hq / pr->hkv;
  if (G > kBwdRows)
    return fail(BA_E_UNSUPPORTED, "hq/hkv > " + std::to_string(kBwdRows) + " unsupported");
  if (!std::isfinite(pr->softmax_scale) || pr->softmax_scale <= 0.f)
    return fail(BA_E_INVAL, "softmax_scale must be finite and positive");
  if (pr->num_groups < 0 || (pr->num_groups > 0 && !pr->groups))
    return fail(BA_E_INVAL, "groups missing");
  if (pr->num_branch_rows < 0) return fail(BA_E_INVAL, "num_branch_rows < 0");

  const int32_t S = pr->num_seqs, C = pr->cp_size, r = pr->cp_rank;
  P.num_seqs = S;
  P.cp_size = C;
  P.cp_rank = r;
  P.hq = pr->hq;
  P.hkv = pr->hkv;
  P.group = G;
  P.head_dim = pr->head_dim;
  P.scale = pr->softmax_scale;
  P.num_branch_rows = pr->num_branch_rows;
  P.cu_seqlens.assign(pr->cu_seqlens, pr->cu_seqlens + S + 1);
  P.n_local = (int64_t)pr->cu_seqlens[S] / C;

  // --- validate groups
  std::vector<uint8_t> used((size_t)pr->num_branch_rows, 0);
  std::vector<std::vector<int32_t>> groups_of_seq(S);
  for (int32_t g = 0; g < pr->num_groups; ++g) {
    const ba_group& gr = pr->groups[g];
    std::string at = "group " + std::to_string(g) + ": ";
    if (gr.seq < 0 || gr.seq >= S) return fail(BA_E_INVAL, at + "seq out of range");
    int32_t L = pr->cu_seqlens[gr.seq + 1] - pr->cu_seqlens[gr.seq];
    if (gr.anchor < 0 || gr.anchor >= L) return fail(BA_E_INVAL, at + "anchor outside the sequence");
    int32_t c = L / (2 * C);
    int32_t chunk = gr.anchor / c;
    int32_t owner = std::min(chunk, 2 * C - 1 - chunk);
    if (owner != r) return fail(BA_E_INVAL, at + "anchor is owned by rank " + std::to_string(owner));
    if (gr.kind != BA_KIND_EAGLE_CHAIN && gr.kind != BA_KIND_DFLASH_BLOCK)
      return fail(BA_E_INVAL, at + "unknown kind");
    if (gr.len < 1 || gr.len > BA_MAX_GROUP_LEN) return fail(BA_E_INVAL, at + "len outside [1, 64]");
    if (gr.row_stride < 1) return fail(BA_E_INVAL, at + "row_stride must be >= 1");
    for (int32_t i = 0; i < gr.len; ++i) {
      int64_t row = (int64_t)gr.row0 + (int64_t)i * gr.row_stride;
      if (row < 0 || row >= pr->num_branch_rows) return fail(BA_E_INVAL, at + "member row out of range");
      if (used[row]) return fail(BA_E_INVAL, at + "member rows overlap another group");
      used[row] = 1;
    }
    groups_of_seq[gr.seq].push_back(g);
  }
  P.groups.resize(pr->num_groups);
  for (int32_t g = 0; g < pr->num_groups; ++g) {
    P.groups[g] = GroupInfo{pr->groups[g].row0, pr->groups[g].row_stride, pr->groups[g].len,
                            pr->groups[g].kind, -1, pr->groups[g].anchor, {0, 0}};
    P.max_group_len = std::max(P.max_group_len, pr->groups[g].len);
  }

  // --- per sequence: token list ordered by causal limit
  P.seqs.resize(S);
  double pairs = 0.0, main_pairs = 0.0;
  int64_t local_off = 0;
  for (int32_t s = 0; s < S; ++s) {
    int32_t L = pr->cu_seqlens[s + 1] - pr->cu_seqlens[s];
    int32_t c = L / (2 * C);
    SeqInfo& si = P.seqs[s];
    si.seg_off = (int32_t)local_off;
    si.c = c;
    si.tok_begin = (int32_t)P.toks.size();
    std::vector<TokInfo> tk;
    bool main_q = pr->has_main ? pr->has_main[s] != 0 : true;
    if (main_q && c > 0) {
      P.any_main_query = true;
      for (int32_t u = 0; u < 2 * c; ++u) {
        int32_t pos = u < c ? r * c + u : (2 * C - 1 - r) * c + (u - c);
        tk.push_back(TokInfo{(int32_t)(local_off + u), pos, -1, -1});
      }
    }
    for (int32_t g : groups_of_seq[s]) {
      const ba_group& gr = pr->groups[g];
      for (int32_t i = 0; i < gr.len; ++i)
        tk.push_back(TokInfo{-(gr.row0 + i * gr.row_stride) - 1, gr.anchor, g, i});
    }
    std::stable_sort(tk.begin(), tk.end(), [](const TokInfo& a, const TokInfo& b) {
      if (a.P != b.P) return a.P < b.P;
      if (a.grp != b.grp) return a.grp < b.grp;  // main (-1) first, then by group
      return a.gidx < b.gidx;
    });
    for (const TokInfo& t : tk) {
      pairs += (double)t.P + 1.0;
      main_pairs += (double)t.P + 1.0;
      if (t.grp >= 0) {
        const ba_group& gr = pr->groups[t.grp];
        pairs += gr.kind == BA_KIND_EAGLE_CHAIN ? (double)(t.gidx + 1) : (double)gr.len;
      }
    }
    for (size_t i = 0; i < tk.size(); ++i)
      if (tk[i].grp >= 0 && tk[i].gidx == 0) P.groups[tk[i].grp].tok0 = (int32_t)(P.toks.size() + i);
    P.toks.insert(P.toks.end(), tk.begin(), tk.end());
    si.tok_end = (int32_t)P.toks.size();
    local_off += 2 * c;
  }
  P.pairs_per_head = pairs;
  P.main_pairs_per_head = main_pairs;

  // --- forward tiles: kFwdRows / G tokens x G heads, never across sequences
  const int32_t tpt = kFwdRows / G;
  struct Keyed {
    int64_t work;
    FwdTile t;
  };
  std::vector<Keyed> ft;
  P.br_keys.clear();
  P.tok_bslot.assign(P.toks.size(), -1);
  for (int32_t s = 0; s < S; ++s) {
    const SeqInfo& si = P.seqs[s];
    for (int32_t t0 = si.tok_begin; t0 < si.tok_end; t0 += tpt) {
      int32_t n = std::min(tpt, si.tok_end - t0);
      int64_t work = (int64_t)P.toks[t0 + n - 1].P + 1;
      // the branch-local keys the tile's tokens attend, each group's once:
      // an EAGLE chain's members 0 .. (deepest member in the tile), a DFlash
      // block's whole block (shared by every KV head's tile)
      std::vector<std::pair<int32_t, int32_t>> need;  // (group, keys)
      for (int32_t t = t0; t < t0 + n; ++t) {
        const TokInfo& tk = P.toks[t];
        if (tk.grp < 0) continue;
        const GroupInfo& g = P.groups[tk.grp];
        const int32_t k = g.kind == BA_KIND_EAGLE_CHAIN ? tk.gidx + 1 : g.len;
        auto it = std::find_if(need.begin(), need.end(), [&](const auto& x) { return x.first == tk.grp; });
        if (it == need.end()) need.emplace_back(tk.grp, k);
        else it->second = std::max(it->second, k);
      }
      int32_t total = 0;
      for (const auto& x : need) total += x.second;
      int32_t bk_off = (int32_t)P.br_keys.size(), bk_n = total;
      if (total > kBrSlots) {
        bk_n = -1;  // the epilogue reads these keys from global memory
      } else {
        int32_t slot = 0;
        for (const auto& x : need) {
          const GroupInfo& g = P.groups[x.first];
          for (int32_t t = t0; t < t0 + n; ++t)
            if (P.toks[t].grp == x.first) P.tok_bslot[t] = slot;
          for (int32_t b = 0; b < x.second; ++b) P.br_keys.push_back(g.row0 + b * g.stride);
          slot += x.second;
        }
      }
      for (int32_t h = 0; h < pr->hkv; ++h) ft.push_back(Keyed{work, FwdTile{s, t0, n, h, bk_off, bk_n}});
    }
  }
  // longest first: the causal prefix length is the tile's work
  std::stable_sort(ft.begin(), ft.end(), [](const Keyed& a, const Keyed& b) { return a.work > b.work; });
  P.fwd_tiles.reserve(ft.size());
  for (auto& k : ft) P.fwd_tiles.push_back(k.t);

  // --- backward tiles: kBwdKeys keys of one ring-step block, grouped by ring
  // step in the order the ring delivers the blocks (step i brings rank
  // (r - i) mod C), longest first inside a step
  P.bwd_step_off.assign(C + 1, 0);
  for (int32_t i = 0; i < C; ++i) {
    const int32_t j = ((r - i) % C + C) % C;
    struct KeyedB {
      int64_t work;
      BwdTile t;
    };
    std::vector<KeyedB> bt;
    for (int32_t s = 0; s < S; ++s) {
      const SeqInfo& si = P.seqs[s];
      if (si.tok_end == si.tok_begin) continue;
      for (int32_t u0 = 0; u0 < 2 * si.c; u0 += kBwdKeys) {
        const int32_t nk = std::min(kBwdKeys, 2 * si.c - u0);
        // tokens are ordered by P and visible_keys is monotone in P
        auto first_with = [&](int32_t need) {
          int32_t lo = si.tok_begin, hi = si.tok_end;
          while (lo < hi) {
            int32_t mid = lo + (hi - lo) / 2;
            if (visible_keys(P.toks[mid].P, j, C, si.c) >= need) hi = mid; else lo = mid + 1;
          }
          return lo;
        };
        const int32_t qb = first_with(u0 + 1);
        const int32_t qf = first_with(u0 + nk);
        if (qb == si.tok_end) continue;
        for (int32_t h = 0; h < pr->hkv; ++h)
          bt.push_back(KeyedB{(int64_t)(si.tok_end - qb),
                              BwdTile{j, s, h, u0, nk, qb, qf, si.tok_end, -1, 0, {0, 0}}});
      }
    }
    // few items: split the longest along their query range (whole 64-row
    // query tiles per piece) into pieces of about total / kKvSplitBelow
    if (!bt.empty() && (int32_t)bt.size() < kKvSplitBelow) {
      const int32_t qt = kBwdRows / G;  // tokens per 64-row query tile
      int64_t total = 0;
      for (const auto& k : bt) total += (k.t.q_end - k.t.q_begin + qt - 1) / qt;
      const int64_t piece = std::max<int64_t>(kKvSplitMinTiles, (total + kKvSplitBelow - 1) / kKvSplitBelow);
      std::vector<KeyedB> split;
      for (const auto& k : bt) {
        const int64_t nt = (k.t.q_end - k.t.q_begin + qt - 1) / qt;
        const int64_t parts = (nt + piece - 1) / piece;
        if (parts < 2) {
          split.push_back(k);
          continue;
        }
        const int32_t slot0 = P.kv_slots;
        const int32_t seg_off = P.seqs[k.t.seq].seg_off;
        P.kv_splits.push_back(KvSplit{k.t.step, seg_off + k.t.u0, k.t.kvh, k.t.nk, slot0, (int32_t)parts, {0, 0}});
        P.kv_slots += (int32_t)parts;
        for (int64_t q = 0; q < parts; ++q) {
          BwdTile t = k.t;
          const int64_t t0 = q * nt / parts, t1 = (q + 1) * nt / parts;
          t.q_begin = k.t.q_begin + (int32_t)(t0 * qt);
          t.q_end = std::min<int32_t>(k.t.q_end, k.t.q_begin + (int32_t)(t1 * qt));
          t.q_full = std::min(std::max(k.t.q_full, t.q_begin), t.q_end);
          t.slot = slot0 + (int32_t)q;
          split.push_back(KeyedB{(int64_t)(t.q_end - t.q_begin), t});
        }
      }
      bt.swap(split);
    }
    std::stable_sort(bt.begin(), bt.end(), [](const KeyedB& a, const KeyedB& b) { return a.work > b.work; });
    // Walk directions for L2 sharing of the Q and dO tiles.  Every item's
    // query range ends at its sequence's last token, and in this longest-
    // first order the lengths of a round of kKvRoundItems items fall about
    // linearly, so the items of an even round start together (those of
    // round 0 at the launch, later ones as a whole previous pair of rounds
    // ends) and walk from the last tile down in step, while an odd round's
    // items start one after another, each as early as its range is long,
    // and walking from their first tile up are in step too.
    for (size_t n = 0; n < bt.size(); ++n) bt[n].t.walk_down = (n / kKvRoundItems) % 2 == 0 ? 1 : 0;
    for (auto& k : bt) P.bwd_tiles.push_back(k.t);
    P.bwd_step_off[i + 1] = (int32_t)P.bwd_tiles.size();
  }
  // the fused schedule: with dK/dV launched per ring step in both schedules
  // and the branch-local keys staged in LDS, it is the faster one on every
  // measured share (the forward and dQ skip the per-step running sums and
  // their finalize passes): 256K share -0.7 %, 32K DFlash sequence -0.9 %,
  // shares of short sequences more
  P.auto_mode = BA_MODE_FUSED;

  pack_image(P);
  return BA_OK;
}

void pack_image(Plan& P) {
  P.image.clear();
  P.off_seqs = append(P.image, P.seqs);
  // the token table is followed by a sentinel whose causal limit -1 admits
  // no key: kernels point rows without a token at it
  std::vector<TokInfo> toks_img(P.toks);
  toks_img.push_back(TokInfo{0, -1, -1, 0});
  P.off_toks = append(P.image, toks_img);
  P.off_groups = append(P.image, P.groups);
  P.off_fwd = append(P.image, P.fwd_tiles);
  P.off_br_keys = append(P.image, P.br_keys);
  P.off_bslot = append(P.image, P.tok_bslot);
  P.off_bwd = append(P.image, P.bwd_tiles);
  P.off_splits = append(P.image, P.kv_splits);
  if (P.rope_theta > 0.f) {
    P.off_pos_block = append(P.image, P.pos_block);
    P.off_pos_qmain = append(P.image, P.pos_qmain);
    P.off_pos_br = append(P.image, P.pos_br);
    P.off_freq = append(P.image, P.rope_freq);
    P.off_rad = append(P.image, P.rope_rad);
  }
  P.image.resize((P.image.size() + 255) & ~size_t(255));
}

// Rotary embedding tables: the position of every row of every ring-step
// block (rank j's local order: chunk j, then chunk 2C-1-j of each sequence)
// and of every branch row (anchor + 1 + member index), and the frequency of
// each of the 64 dim pairs in turns per position.
void rope_freq_table(float theta, RopeFreq* out) {
  const double two_pi = 6.283185307179586476925286766559;
  for (int j = 0; j < kHeadDim / 2; ++j) {
    const double f = std::pow((double)theta, -(double)j / (kHeadDim / 2)) / two_pi;
    const float hi = (float)f;
    out[j] = RopeFreq{hi, (float)(f - (double)hi)};
  }
}

void rope_rad_table(float theta, double* out) {
  for (int j = 0; j < kHeadDim / 2; ++j) out[j] = std::pow((double)theta, -(double)j / (kHeadDim / 2));
}

static int build_rope(Plan& P, float theta) {
  if (!std::isfinite(theta) || theta < 0.f) return fail(BA_E_INVAL, "rope theta must be finite and >= 0");
  P.rope_theta = theta;
  P.pos_block.clear();
  P.pos_qmain.clear();
  P.pos_br.clear();
  P.rope_freq.clear();
  P.rope_rad.clear();
  if (theta > 0.f) {
    const int32_t C = P.cp_size;
    int64_t max_pos = 0;
    P.pos_block.resize((size_t)C * P.n_local);
    for (int32_t j = 0; j < C; ++j)
      for (int32_t s = 0; s < P.num_seqs; ++s) {
        const SeqInfo& si = P.seqs[s];
        for (int32_t u = 0; u < 2 * si.c; ++u) {
          const int32_t pos = u < si.c ? j * si.c + u : (2 * C - 1 - j) * si.c + (u - si.c);
          P.pos_block[(size_t)j * P.n_local + si.seg_off + u] = pos;
          max_pos = std::max<int64_t>(max_pos, pos);
        }
      }
    P.pos_qmain.assign((size_t)P.n_local, -1);
    for (const TokInfo& t : P.toks)
      if (t.qrow >= 0) P.pos_qmain[t.qrow] = P.pos_block[(size_t)P.cp_rank * P.n_local + t.qrow];
    P.pos_br.assign((size_t)P.num_branch_rows, -1);
    for (const GroupInfo& g : P.groups)
      for (int32_t i = 0; i < g.len; ++i) {
        P.pos_br[(size_t)g.row0 + (size_t)i * g.stride] = g.anchor + 1 + i;
        max_pos = std::max<int64_t>(max_pos, (int64_t)g.anchor + 1 + i);
      }
    if (max_pos >= (1 << 24)) {
      P.rope_theta = 0.f;
      P.pos_block.clear();
      P.pos_qmain.clear();
      P.pos_br.clear();
      pack_image(P);
      return fail(BA_E_UNSUPPORTED, "rope positions must stay below 2^24");
    }
    P.rope_freq.resize(kHeadDim / 2);
    rope_freq_table(theta, P.rope_freq.data());
    P.rope_rad.resize(kHeadDim / 2);
    rope_rad_table(theta, P.rope_rad.data());
  }
  pack_image(P);
  return BA_OK;
}

}  // namespace ba

extern "C" {

const char* branch_attn_last_error(void) { return ba::g_last_error.c_str(); }

int zigzag_partition(const int32_t* cu_seqlens, int32_t num_seqs, int32_t cp_size, int32_t cp_rank,
                     int32_t* local_cu_seqlens, int32_t* local_to_global, int32_t* local_pos) {
  int rc = ba::check_seqlens(cu_seqlens, num_seqs, cp_size, cp_rank);
  if (rc) return rc;
  if (!local_cu_seqlens || !local_to_global || !local_pos)
    return ba::fail(BA_E_INVAL, "output arrays must not be NULL");
  const int32_t C = cp_size, r = cp_rank;
  int64_t out = 0;
  local_cu_seqlens[0] = 0;
  for (int32_t s = 0; s < num_seqs; ++s) {
    int32_t L = cu_seqlens[s + 1] - cu_seqlens[s];
    int32_t c = L / (2 * C);
    for (int32_t half = 0; half < 2; ++half) {
      int32_t chunk = half == 0 ? r : 2 * C - 1 - r;
      for (int32_t i = 0; i < c; ++i) {
        int32_t pos = chunk * c + i;
        local_pos[out] = pos;
        local_to_global[out] = cu_seqlens[s] + pos;
        ++out;
      }
    }
    local_cu_seqlens[s + 1] = (int32_t)out;
  }
  return BA_OK;
}

int branch_attn_plan_create(const ba_problem* prob, ba_plan** out) {
  if (!out) return ba::fail(BA_E_INVAL, "out is NULL");
  *out = nullptr;
  if (!prob) return ba::fail(BA_E_INVAL, "problem is NULL");
  ba_plan* p = new (std::nothrow) ba_plan();
  if (!p) return ba::fail(BA_E_INVAL, "out of host memory");
  int rc;
  try {
    rc = ba::build_plan(prob, p->p);
  } catch (const std::exception& e) {
    rc = ba::fail(BA_E_INVAL, std::string("plan construction failed: ") + e.what());
  }
  if (rc) {
    delete p;
    return rc;
  }
  *out = p;
  return BA_OK;
}

void branch_attn_plan_destroy(ba_plan* plan) { delete plan; }

int branch_attn_plan_set_rope(ba_plan* plan, float theta) {
  if (!plan) return ba::fail(BA_E_INVAL, "plan is NULL");
  try {
    return ba::build_rope(plan->p, theta);
  } catch (const std::exception& e) {
    return ba::fail(BA_E_INVAL, std::string("rope tables: ") + e.what());
  }
}

int branch_attn_plan_positions(const ba_plan* plan, int32_t* main_pos, int32_t* br_pos) {
  if (!plan) return ba::fail(BA_E_INVAL, "plan is NULL");
  const ba::Plan& P = plan->p;
  if (main_pos) {
    const int32_t C = P.cp_size, r = P.cp_rank;
    for (int32_t s = 0; s < P.num_seqs; ++s) {
      const ba::SeqInfo& si = P.seqs[s];
      for (int32_t u = 0; u < 2 * si.c; ++u)
        main_pos[si.seg_off + u] = u < si.c ? r * si.c + u : (2 * C - 1 - r) * si.c + (u - si.c);
    }
  }
  if (br_pos) {
    for (int32_t i = 0; i < P.num_branch_rows; ++i) br_pos[i] = -1;
    for (const ba::GroupInfo& g : P.groups)
      for (int32_t i = 0; i < g.len; ++i) br_pos[(size_t)g.row0 + (size_t)i * g.stride] = g.anchor + 1 + i;
  }
  return BA_OK;
}

int branch_attn_plan_mode(const ba_plan* plan, int32_t mode, int32_t* resolved) {
  if (!plan) return ba::fail(BA_E_INVAL, "plan is NULL");
  if (mode != BA_MODE_PER_STEP && mode != BA_MODE_FUSED && mode != BA_MODE_AUTO)
    return ba::fail(BA_E_INVAL, "unknown mode");
  if (resolved) *resolved = ba::resolve_mode(plan->p, mode);
  return BA_OK;
}

int branch_attn_workspace_size(const ba_plan* plan, int32_t mode, size_t* fwd_bytes, size_t* bwd_bytes) {
  if (!plan) return ba::fail(BA_E_INVAL, "plan is NULL");
  if (mode != BA_MODE_PER_STEP && mode != BA_MODE_FUSED && mode != BA_MODE_AUTO)
    return ba::fail(BA_E_INVAL, "unknown mode");
  mode = ba::resolve_mode(plan->p, mode);
  ba::WorkspaceLayout w = ba::workspace_layout(plan->p, mode);
  if (fwd_bytes) *fwd_bytes = w.fwd_total;
  if (bwd_bytes) *bwd_bytes = w.bwd_total;
  return BA_OK;
}

int branch_attn_plan_info(const ba_plan* plan, int64_t* n_local, int64_t* n_query_tokens) {
  if (!plan) return ba::fail(BA_E_INVAL, "plan is NULL");
  if (n_local) *n_local = plan->p.n_local;
  if (n_query_tokens) *n_query_tokens = (int64_t)plan->p.toks.size();
  return BA_OK;
}

int branch_attn_useful_flops(const ba_plan* plan, double* fwd_flops, double* bwd_flops) {
  if (!plan) return ba::fail(BA_E_INVAL, "plan is NULL");
  const ba::Plan& p = plan->p;
  double per = p.pairs_per_head * p.hq * p.head_dim;
  if (fwd_flops) *fwd_flops = 4.0 * per;
  if (bwd_flops) *bwd_flops = 10.0 * per;
  return BA_OK;
}

int branch_attn_pair_counts(const ba_plan* plan, double* main_pairs, double* local_pairs) {
  if (!plan) return ba::fail(BA_E_INVAL, "plan is NULL");
  if (main_pairs) *main_pairs = plan->p.main_pairs_per_head;
  if (local_pairs) *local_pairs = plan->p.pairs_per_head - plan->p.main_pairs_per_head;
  return BA_OK;
}

}  // extern "C"
