// Host-side fuzz of the plan builder and the host entry points of the C ABI,
// built with AddressSanitizer and UndefinedBehaviorSanitizer (host code
// only, no GPU): seeded random problems, valid and malformed (anchors on
// other ranks or past the sequence, bad group lengths, overlapping or
// out-of-range member rows, bad kinds, strides, head sizes, scales and
// lengths), each run through zigzag_partition, plan creation and every host
// query of a plan.  Any invalid memory access or undefined behaviour aborts
// the run; a valid problem that is rejected, or a malformed one that is
// accepted, fails it.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "branch_attn.h"

namespace {

std::mt19937_64 rng(20261202);
int uni(int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); }  // inclusive
bool coin(double p) { return std::uniform_real_distribution<double>(0.0, 1.0)(rng) < p; }

int fails = 0;
void expect(bool ok, const char* what, int iter, int rc) {
  if (!ok) {
    std::fprintf(stderr, "iteration %d: %s (rc %d: %s)\n", iter, what, rc, branch_attn_last_error());
    ++fails;
  }
}

int owner(int p, int c, int C) {
  const int chunk = p / c;
  return chunk < 2 * C - 1 - chunk ? chunk : 2 * C - 1 - chunk;
}

}  // namespace

int main(int argc, char** argv) {
  const int iters = argc > 1 ? std::atoi(argv[1]) : 3000;
  int accepted = 0, rejected = 0;
  for (int it = 0; it < iters; ++it) {
    const int cps[] = {1, 2, 3, 4, 8};
    const int C = cps[uni(0, 4)], r = uni(0, C - 1), S = uni(1, 4);
    std::vector<int32_t> cu(S + 1, 0);
    for (int s = 0; s < S; ++s) cu[s + 1] = cu[s] + 2 * C * (coin(0.1) ? uni(100, 2000) : uni(0, 24));
    bool bad = false;
    if (coin(0.03)) {  // a length that is not a multiple of 2C
      for (int s = 1; s <= S; ++s) cu[s] += 1;
      bad = true;
    }
    const int N = cu[S];
    // zigzag_partition on its own
    {
      const int nl = N / C + 1;
      std::vector<int32_t> lcu(S + 1), l2g(nl), lp(nl);
      const int rr = coin(0.05) ? C : r;
      const int rc = zigzag_partition(cu.data(), S, C, rr, lcu.data(), l2g.data(), lp.data());
      expect((rc == BA_OK) == (!bad && rr == r), "zigzag_partition verdict", it, rc);
    }
    std::vector<uint8_t> has_main(S);
    for (auto& h : has_main) h = coin(0.7);
    const int heads[][2] = {{1, 1}, {4, 2}, {8, 1}, {32, 8}, {6, 3}};
    const int hi = uni(0, 4);
    int hq = heads[hi][0], hkv = heads[hi][1], hd = 128;
    float scale = 0.0883883f;
    if (coin(0.02)) { hd = 64; bad = true; }
    if (coin(0.02)) { scale = std::nanf(""); bad = true; }
    if (coin(0.02)) { hq = 5; hkv = 2; bad = true; }
    // groups anchored on the rank's own positions
    std::vector<ba_group> g;
    int rows = 0;
    for (int s = 0; s < S && !bad; ++s) {
      const int L = cu[s + 1] - cu[s], c = L / (2 * C);
      if (c == 0) continue;
      const int ng = uni(0, 6);
      for (int k = 0; k < ng; ++k) {
        int p = uni(0, L - 1);
        for (int t = 0; t < 8 && owner(p, c, C) != r; ++t) p = uni(0, L - 1);
        if (owner(p, c, C) != r) continue;
        const int kind = coin(0.5) ? BA_KIND_EAGLE_CHAIN : BA_KIND_DFLASH_BLOCK;
        const int len = uni(1, kind == BA_KIND_EAGLE_CHAIN ? 8 : 32);
        g.push_back(ba_group{s, p, kind, len, rows, 1});
        rows += len;
      }
    }
    int nrows = rows;
    if (!bad && coin(0.25)) {  // one malformation
      const int m = uni(0, 8);
      if (m == 0 && !g.empty()) g[0].anchor = cu[g[0].seq + 1] - cu[g[0].seq];  // past the end
      else if (m == 1 && !g.empty()) g[0].len = 0;
      else if (m == 2 && !g.empty()) g[0].len = 65;
      else if (m == 3 && !g.empty()) g[0].row0 = -1;
      else if (m == 4 && g.size() > 1) g[1].row0 = g[0].row0;  // overlapping members
      else if (m == 5 && !g.empty()) g[0].kind = 7;
      else if (m == 6 && !g.empty()) g[0].row_stride = 0;
      else if (m == 7 && !g.empty()) nrows = rows - 1;  // members past the branch arrays
      else if (m == 8 && !g.empty()) g[0].seq = S;
      bad = !g.empty() && !(m == 4 && g.size() <= 1);
    }
    if (!bad && C > 1 && !g.empty() && coin(0.05)) {  // anchor on a position of another rank
      const ba_group& g0 = g[0];
      const int L = cu[g0.seq + 1] - cu[g0.seq], c = L / (2 * C);
      for (int p = 0; p < L; ++p)
        if (owner(p, c, C) != r) {
          g[0].anchor = p;
          bad = true;
          break;
        }
    }
    ba_problem prob{S, cu.data(), has_main.data(), C, r, hq, hkv, hd, scale, (int32_t)g.size(),
                    g.empty() ? nullptr : g.data(), nrows};
    ba_plan* plan = nullptr;
    const int rc = branch_attn_plan_create(&prob, &plan);
    expect((rc == BA_OK) == !bad, bad ? "malformed problem accepted" : "valid problem rejected", it, rc);
    if (rc != BA_OK) {
      expect(plan == nullptr, "failed create left a plan", it, rc);
      ++rejected;
      continue;
    }
    ++accepted;
    int64_t n_local = -1, ntok = -1;
    expect(branch_attn_plan_info(plan, &n_local, &ntok) == BA_OK && n_local == N / C, "plan_info", it, 0);
    std::vector<int32_t> mp(n_local + 1), bp(nrows + 1);
    expect(branch_attn_plan_positions(plan, mp.data(), bp.data()) == BA_OK, "positions", it, 0);
    for (const ba_group& gr : g)
      for (int i = 0; i < gr.len; ++i)
        expect(bp[gr.row0 + i * gr.row_stride] == gr.anchor + 1 + i, "branch position", it, 0);
    size_t f0, b0, f1, b1;
    expect(branch_attn_workspace_size(plan, BA_MODE_PER_STEP, &f0, &b0) == BA_OK &&
               branch_attn_workspace_size(plan, BA_MODE_FUSED, &f1, &b1) == BA_OK,
           "workspace sizes", it, 0);
    double a, b;
    expect(branch_attn_useful_flops(plan, &a, &b) == BA_OK && a >= 0 && b >= 0, "useful flops", it, 0);
    expect(branch_attn_pair_counts(plan, &a, &b) == BA_OK && a >= 0 && b >= 0, "pair counts", it, 0);
    expect(branch_attn_plan_set_rope(plan, 1.0e4f) == BA_OK, "set_rope", it, 0);
    size_t f2, b2;
    expect(branch_attn_workspace_size(plan, BA_MODE_PER_STEP, &f2, &b2) == BA_OK && f2 >= f0 && b2 >= b0,
           "rope workspace", it, 0);
    expect(branch_attn_plan_set_rope(plan, 0.0f) == BA_OK, "rope off", it, 0);
    branch_attn_plan_destroy(plan);
  }
  std::printf("plan fuzz: %d iterations, %d accepted, %d rejected, %d failures\n", iters, accepted, rejected, fails);
  return fails ? 1 : 0;
}
