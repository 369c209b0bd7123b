// Randomised checks of libchunk's host core: the Order generators, Order
// validation and flattening, the canonical parameter layout and the
// workspace plan, fed random and mostly invalid arguments. Built with the
// host compiler under AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitize.py; a sanitizer report or a failed consistency
// check ends it with a non-zero status.
#include <stdio.h>
#include <stdlib.h>

#include <random>
#include <vector>

#include "host_core.hpp"

using namespace lc;

#define CHECK(c)                                                           \
  do {                                                                     \
    if (!(c)) {                                                            \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c);      \
      return 1;                                                            \
    }                                                                      \
  } while (0)

int main(int argc, char **argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 20000;
  std::mt19937 rng(20260);
  auto rnd = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  int generated = 0, valid_random = 0, plans = 0;
  for (int it = 0; it < iters; ++it) {
    // generators with random arguments and capacities; what they return
    // must pass validation and flatten to the same length
    const int M = rnd(-2, 40), P = rnd(-1, 12), s = rnd(-1, 12), wd = rnd(-1, 12);
    const int cap = rnd(-1, 100);
    std::vector<lc_order_entry> buf(cap > 0 ? cap : 1);
    for (int g = 0; g < 3; ++g) {
      int32_t n = -7;
      const lc_status st = g == 0 ? lc_order_1f1b(M, P, s, buf.data(), cap, &n)
                           : g == 1 ? lc_order_1f1b_overlap(M, P, s, buf.data(), cap, &n)
                                    : lc_order_1f1b_split(M, P, s, wd, buf.data(), cap, &n);
      if (st != LC_OK) continue;
      ++generated;
      CHECK(n == 2 * M + (g == 2 ? M : 0) && n <= cap);
      lc_order o{M, n, buf.data()};
      int32_t peak = -1, peak_w = -1;
      CHECK(lc_order_validate_split(&o, M, M, &peak, &peak_w) == LC_OK);
      CHECK(peak >= 1 && peak <= M && peak_w >= 0 && peak_w <= M);
      std::vector<lc_order_entry> flat;
      CHECK(flatten_order(o, &flat) == LC_OK);
      CHECK((int)flat.size() == n);
    }
    // random entry lists, mostly invalid: no read outside them, and what
    // validates also flattens
    const int ne = rnd(0, 30);
    std::vector<lc_order_entry> e(ne > 0 ? ne : 1);
    for (int i = 0; i < ne; ++i) {
      e[i].mb = rnd(-1, 6);
      int p = rnd(0, 3);
      if (rnd(0, 4) == 0) p |= LC_ORDER_WITH_NEXT;
      if (rnd(0, 50) == 0) p = rnd(-5, 600);
      e[i].pass = p;
    }
    lc_order o{rnd(-1, 6), ne, ne ? e.data() : nullptr};
    int32_t peak = 0, peak_w = 0;
    if (lc_order_validate_split(&o, rnd(-1, 6), rnd(-1, 6), &peak, &peak_w) == LC_OK) {
      ++valid_random;
      std::vector<lc_order_entry> flat;
      const lc_status fs = flatten_order(o, &flat);
      CHECK(fs == LC_OK && (int)flat.size() == ne);
    }
    // random valid Orders: F and B (or Bi, with its Bw anywhere later)
    // subsequences each in microbatch order, randomly merged, then random
    // overlap flags; validation decides, flattening must agree
    {
      const int m = rnd(1, 8);
      const bool sp = rnd(0, 1);
      std::vector<lc_order_entry> ord;
      std::vector<int> pending;  // microbatches whose Bw is still to place
      int nf = 0, nb = 0;
      while (nf < m || nb < m || !pending.empty()) {
        const int c = rnd(0, 2);
        if (c == 0 && nf < m) {
          ord.push_back({nf++, LC_PASS_F});
        } else if (c == 1 && nb < nf) {
          ord.push_back({nb, sp ? LC_PASS_BI : LC_PASS_B});
          if (sp) pending.push_back(nb);
          ++nb;
        } else if (c == 2 && !pending.empty()) {
          const int k = rnd(0, (int)pending.size() - 1);
          ord.push_back({pending[k], LC_PASS_BW});
          pending.erase(pending.begin() + k);
        }
      }
      for (size_t i = 0; i + 1 < ord.size(); ++i)
        if (rnd(0, 3) == 0) ord[i].pass |= LC_ORDER_WITH_NEXT;
      lc_order ov{m, (int32_t)ord.size(), ord.data()};
      int32_t pk = 0, pw = 0;
      const lc_status vs2 = lc_order_validate_split(&ov, m, m, &pk, &pw);
      std::vector<lc_order_entry> flat;
      const lc_status fs2 = flatten_order(ov, &flat);
      if (vs2 == LC_OK) {
        ++valid_random;
        CHECK(fs2 == LC_OK && flat.size() == ord.size());
      }
    }
    // descriptors with random fields, some far out of range
    lc_stage_desc d{};
    d.n_layers = rnd(-1, 6);
    d.head_dim = 16 << rnd(0, 3);
    d.n_heads = rnd(0, 8);
    d.d_model = rnd(0, 5) == 0 ? rnd(-3, 1 << 20) : d.n_heads * d.head_dim;
    d.n_kv_heads = rnd(0, 3) == 0 ? rnd(-1, 8) : 0;
    d.qk_norm = rnd(0, 1);
    d.n_experts = rnd(0, 2) == 0 ? rnd(-1, 70) : 0;
    d.top_k = rnd(1, 3);
    d.d_ff = 64 * rnd(-1, 200);
    d.d_ff_expert = 64 * rnd(-1, 40);
    d.seq_len = 128 * rnd(-1, 64);
    d.micro_batch = rnd(-1, 4);
    d.rms_eps = 1e-5f;
    d.rope_base = 10000.0f;
    d.causal = rnd(0, 10) == 0 ? 0 : 1;
    d.compute_dtype = rnd(-1, 2);
    size_t bytes = 0;
    const int mif = rnd(-1, 4), mwp = rnd(-1, 4);
    if (lc_workspace_bytes_split(&d, mif, mwp, &bytes) == LC_OK) {
      ++plans;
      StagePlan sp{};
      CHECK(stage_plan(d, mif, mwp, &sp) == LC_OK);
      CHECK(sp.slot0 + sp.slot_bytes * (size_t)mif <= bytes);
      CHECK(sp.wslot0 + sp.wslot_bytes * (size_t)mwp <= bytes);
      CHECK(sp.wlayer_bytes * (size_t)d.n_layers == sp.wslot_bytes);
      size_t np = 0;
      CHECK(lc_param_count(&d, &np) == LC_OK);
      // every tensor of every layer (and expert) lies inside the bucket
      for (int layer = 0; layer < d.n_layers; ++layer)
        for (int tid = LC_T_WQ; tid <= LC_T_KN; ++tid)
          for (int ex = 0; ex < (d.n_experts > 0 ? d.n_experts : 1); ++ex) {
            size_t off = 0;
            int64_t shape[2] = {0, 0};
            if (lc_param_offset(&d, layer, tid, ex, &off, shape) != LC_OK) continue;
            CHECK(shape[0] > 0 && shape[1] > 0);
            CHECK(off + (size_t)(shape[0] * shape[1]) <= np);
          }
      size_t o2 = 0;
      int64_t sh[2];
      CHECK(lc_param_offset(&d, d.n_layers, LC_T_WQ, 0, &o2, sh) != LC_OK);
      CHECK(lc_param_offset(&d, 0, 99, 0, &o2, sh) != LC_OK);
    }
  }
  printf("ok: %d iterations, %d generated Orders, %d valid random Orders, %d plans\n", iters,
         generated, valid_random, plans);
  return 0;
}
