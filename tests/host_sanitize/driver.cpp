// Host-only driver for the sanitizer build of the library's host code (planner.cpp and
// host_checks.cpp, compiled with g++ -fsanitize=address,undefined): exercises every host entry
// point on valid, boundary and invalid arguments and checks the documented status codes. Exits 0
// when every check holds; any sanitizer report aborts with a non-zero status.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <limits>
#include <string>
#include <vector>

#include "ditplan.h"
#include "ditstep.h"
#include "host_checks.h"

static int failures = 0;
#define CHECK(cond)                                                        \
  do {                                                                     \
    if (!(cond)) {                                                         \
      std::fprintf(stderr, "%s:%d check failed: %s\n", __FILE__, __LINE__, #cond); \
      failures++;                                                          \
    }                                                                      \
  } while (0)

static dit_block_config cfg(int hidden, int heads, int hd, int mlp, int n_img, int n_txt, int gh, int gw) {
  dit_block_config c{};
  c.hidden = hidden; c.heads = heads; c.head_dim = hd; c.mlp_hidden = mlp;
  c.n_img = n_img; c.n_txt = n_txt; c.grid_h = gh; c.grid_w = gw;
  c.rope = 1; c.ln_eps = 1e-6f; c.rope_theta = 1e4f; c.dtype = DIT_BF16;
  return c;
}

static void status_text() {
  for (int s = 0; s <= 8; s++) CHECK(std::strlen(dit_status_string((dit_status)s)) > 0);
  CHECK(dit_abi_version() == DIT_ABI_VERSION);
}

static void config_checks() {
  dit_block_config c = cfg(3072, 24, 128, 12288, 1024, 256, 32, 32);
  CHECK(dit::check_config(&c) == DIT_OK);
  CHECK(dit::check_config(nullptr) == DIT_ERR_INVALID_ARG);
  dit_block_config b = c; b.head_dim = 100;
  CHECK(dit::check_config(&b) == DIT_ERR_SHAPE);
  b = c; b.n_img = 1023;
  CHECK(dit::check_config(&b) == DIT_ERR_SHAPE);
  b = c; b.hidden = 8192; b.heads = 64;
  CHECK(dit::check_config(&b) == DIT_ERR_UNSUPPORTED);
  b = c; b.ln_eps = std::numeric_limits<float>::quiet_NaN();
  CHECK(dit::check_config(&b) == DIT_ERR_INVALID_ARG);
  b = c; b.dtype = 7;
  CHECK(dit::check_config(&b) == DIT_ERR_INVALID_ARG);
  b = c; b.grid_h = std::numeric_limits<int32_t>::max(); b.grid_w = 2;   // product overflows int32
  CHECK(dit::check_config(&b) != DIT_OK);
  CHECK(std::strlen(dit_last_error_message()) > 0);
}

static void flow_checks() {
  float cx, cv, ce;
  CHECK(dit::flow_coefficients(0.5f, 0.45f, 0.f, false, &cx, &cv, &ce) == DIT_OK && cx == 1.f && ce == 0.f);
  CHECK(dit::flow_coefficients(0.5f, 0.45f, 0.7f, true, &cx, &cv, &ce) == DIT_OK && ce > 0.f);
  CHECK(dit::flow_coefficients(0.5f, 0.55f, 0.f, false, &cx, &cv, &ce) == DIT_ERR_DOMAIN);
  CHECK(dit::flow_coefficients(1.0f, 0.95f, 0.7f, true, &cx, &cv, &ce) == DIT_ERR_DOMAIN);
  CHECK(dit::flow_coefficients(0.5f, 0.45f, 0.7f, false, &cx, &cv, &ce) == DIT_ERR_INVALID_ARG);
  CHECK(dit::flow_coefficients(NAN, 0.45f, 0.f, false, &cx, &cv, &ce) == DIT_ERR_DOMAIN);
  CHECK(dit::flow_coefficients(0.5f, 0.45f, -1.f, false, &cx, &cv, &ce) == DIT_ERR_DOMAIN);
}

static void teacache_checks() {
  dit_teacache_state st;
  double coef[8] = {1, 2, 3, 4, 5, 6, 7, 8};
  CHECK(dit_teacache_init(&st, 0.3, coef, 8) == DIT_OK);
  CHECK(dit_teacache_init(&st, 0.3, coef, 9) == DIT_ERR_INVALID_ARG);
  CHECK(dit_teacache_init(&st, -1.0, nullptr, 0) == DIT_ERR_INVALID_ARG);
  CHECK(dit_teacache_init(nullptr, 0.3, nullptr, 0) == DIT_ERR_INVALID_ARG);
  CHECK(dit_teacache_init(&st, 0.3, nullptr, 0) == DIT_OK);
  int32_t run = -1;
  CHECK(dit_teacache_gate(&st, 0.1, 0, &run) == DIT_OK && run == 1);   // no previous input yet
  st.has_prev = st.has_residual = 1;
  const double rel[5] = {0.1, 0.15, 0.1, 0.02, 0.25};
  const int want[5] = {0, 0, 1, 0, 0};
  for (int i = 0; i < 5; i++) CHECK(dit_teacache_gate(&st, rel[i], 0, &run) == DIT_OK && run == want[i]);
  CHECK(dit_teacache_gate(&st, NAN, 0, &run) == DIT_ERR_NAN);
  CHECK(dit_teacache_gate(&st, 0.1, 0, nullptr) == DIT_ERR_INVALID_ARG);
  st.n_coef = 42;   // a corrupted state is rejected, not indexed
  CHECK(dit_teacache_gate(&st, 0.1, 0, &run) == DIT_ERR_INVALID_ARG);
}

static void planner_checks() {
  const int32_t dv[4] = {4, 8, 16, 32}, sv[2] = {12, 20};
  dit_planner* p = nullptr;
  CHECK(dit_planner_create(dv, 4, sv, 2, 0.5, 3, 64, &p) == DIT_OK && p);
  CHECK(dit_planner_num_actions(p) == 8);
  int32_t d, s;
  CHECK(dit_planner_action(p, 7, &d, &s) == DIT_OK && d == 32 && s == 20);
  CHECK(dit_planner_action(p, 8, &d, &s) == DIT_ERR_INVALID_ARG);
  CHECK(dit_planner_action(p, -1, &d, &s) == DIT_ERR_INVALID_ARG);
  std::vector<int32_t> el(8);
  int32_t cnt = 0, idx = 0, fits = 0;
  double ucb = 0;
  for (int it = 0; it < 200; it++) {
    const double t_train = 0.5 * (it % 37), t_step = 0.01 + 0.001 * (it % 11);
    const int n_spot = it % 9;
    CHECK(dit_planner_eligible(p, t_train, n_spot, t_step, el.data(), &cnt) == DIT_OK);
    CHECK(dit_planner_select(p, t_train, n_spot, t_step, &idx, &fits, it % 2 ? &ucb : nullptr) == DIT_OK);
    CHECK(idx >= 0 && idx < 8);
    CHECK(dit_planner_update(p, idx, 1.0 + 0.01 * (it % 5)) == DIT_OK);
  }
  int32_t tot, win;
  double mean;
  CHECK(dit_planner_stats(p, 0, &tot, &win, &mean, &ucb) == DIT_OK && win <= 3);
  CHECK(dit_planner_update(p, 8, 1.0) == DIT_ERR_INVALID_ARG);
  CHECK(dit_planner_update(p, 0, INFINITY) != DIT_OK);
  CHECK(dit_planner_select(p, 1.0, 1, 0.0, &idx, &fits, nullptr) == DIT_ERR_DOMAIN);
  CHECK(dit_planner_eligible(p, -1.0, 1, 0.1, el.data(), &cnt) == DIT_ERR_DOMAIN);
  dit_planner_destroy(p);
  dit_planner_destroy(nullptr);
  dit_planner* q = reinterpret_cast<dit_planner*>(0x1);
  const int32_t dup[2] = {8, 8};
  CHECK(dit_planner_create(dup, 2, sv, 2, 0.5, 3, 64, &q) == DIT_ERR_INVALID_ARG && q == nullptr);
  CHECK(dit_planner_create(dv, 0, sv, 2, 0.5, 3, 64, &q) == DIT_ERR_INVALID_ARG);
  CHECK(dit_planner_create(dv, 4, sv, 2, -0.5, 3, 64, &q) == DIT_ERR_INVALID_ARG);
  CHECK(dit_planner_create(dv, 4, sv, 2, 0.5, 0, 64, &q) == DIT_ERR_INVALID_ARG);
  CHECK(dit_planner_create(dv, 4, sv, 2, 0.5, 3, 64, nullptr) == DIT_ERR_INVALID_ARG);
  // feedback
  const float sig[4] = {0.1f, 0.2f, 0.3f, 0.4f};
  const int32_t ex[4] = {1, 0, 1, 0}, all[4] = {1, 1, 1, 1};
  double r = 0;
  CHECK(dit_planner_feedback(sig, ex, 4, &r) == DIT_OK && std::fabs(r - 0.25 / 0.3) < 1e-6);
  CHECK(dit_planner_feedback(sig, all, 4, &r) == DIT_ERR_DOMAIN);
  const float bad[2] = {NAN, 1.f};
  const int32_t none[2] = {0, 0};
  CHECK(dit_planner_feedback(bad, none, 2, &r) == DIT_ERR_NAN);
  CHECK(dit_planner_feedback(sig, ex, 0, &r) != DIT_OK);
}

static void seed_bank_checks() {
  for (int k = 0; k <= 9; k++) {
    dit_seed_bank* b = nullptr;
    CHECK(dit_seed_bank_create(k, &b) == DIT_OK && b);
    for (int dlen = 0; dlen <= 12; dlen++) {
      std::vector<int64_t> seeds(dlen);
      std::vector<float> rw(dlen);
      for (int j = 0; j < dlen; j++) { seeds[j] = 1000 + j; rw[j] = (float)((j * 7) % 4) * 0.25f; }
      CHECK(dit_seed_bank_put(b, dlen, seeds.data(), rw.data(), dlen) == DIT_OK);
      int64_t out[3];
      int32_t cnt = -1;
      CHECK(dit_seed_bank_get(b, dlen, out, 3, &cnt) == DIT_OK && cnt == std::min(k, dlen));
      CHECK(dit_seed_bank_get(b, 999, out, 0, &cnt) == DIT_OK && cnt == 0);
    }
    // put_selected: 3 groups of 6 seeds, positions from a selection of min(k, 6)
    const int g = 3, dd = 6, kk = std::min(k, dd);
    std::vector<int64_t> ids = {7, 8, 9}, seeds(g * dd);
    std::vector<int32_t> sel(g * std::max(kk, 1));
    for (int i = 0; i < g * dd; i++) seeds[i] = 50 + i;
    for (int i = 0; i < g; i++)
      for (int j = 0; j < kk; j++) sel[i * kk + j] = (j * 5 + i) % dd;
    CHECK(dit_seed_bank_put_selected(b, ids.data(), g, seeds.data(), dd, sel.data(), kk) == DIT_OK);
    if (kk > 0) {
      sel[0] = dd;   // out of range
      CHECK(dit_seed_bank_put_selected(b, ids.data(), g, seeds.data(), dd, sel.data(), kk) == DIT_ERR_INVALID_ARG);
    }
    const float nanr[2] = {NAN, 0.f};
    const int64_t s2[2] = {1, 2};
    CHECK(dit_seed_bank_put(b, 1, s2, nanr, 2) == DIT_ERR_NAN);
    CHECK(dit_seed_bank_size(b) >= 1);
    dit_seed_bank_destroy(b);
  }
  dit_seed_bank_destroy(nullptr);
  CHECK(dit_seed_bank_create(-1, nullptr) == DIT_ERR_INVALID_ARG);
}

int main() {
  status_text();
  config_checks();
  flow_checks();
  teacache_checks();
  planner_checks();
  seed_bank_checks();
  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("host sanitizer driver: all checks passed\n");
  return 0;
}
