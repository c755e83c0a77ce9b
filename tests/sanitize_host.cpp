// The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer: argument
// checks, work items, workspace layout and visible-pair counts of the plan on random and
// malformed problems, and the scheduler on random and malformed batches.  Built with g++
// (no GPU code) by tests/test_host_sanitizers.py; any report aborts with a non-zero status.
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "hydra_sched.h"
#include "plan.h"

namespace {

std::mt19937_64 rng(7);

int64_t uni(int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(rng); }

void random_chunk(hydra_chunk_t* c, int32_t total) {
  c->n_segs = int32_t(uni(0, HYDRA_MAX_SEGS));
  for (int s = 0; s < c->n_segs; ++s) {
    const int64_t a = uni(0, total), b = uni(a, total);
    c->start[s] = int32_t(a);
    c->len[s] = int32_t(b - a);
  }
}

}  // namespace

int main() {
  int64_t planned = 0, refused = 0, pairs = 0;
  for (int trial = 0; trial < 4000; ++trial) {
    const int n_docs = int(uni(1, 9));
    std::vector<int32_t> cu(size_t(n_docs) + 1, 0);
    for (int d = 0; d < n_docs; ++d) cu[size_t(d) + 1] = cu[size_t(d)] + int32_t(uni(0, 700));
    hydra_problem_t p{};
    p.n_heads = int32_t(uni(1, 8));
    p.d_qk = 192;
    p.d_v = 128;
    p.cu_seqlens = cu.data();
    p.n_docs = n_docs;
    random_chunk(&p.q, cu.back());
    random_chunk(&p.kv, cu.back());
    // malformed variants
    if (trial % 7 == 1 && p.q.n_segs > 0) p.q.len[0] = -int32_t(uni(1, 5));
    if (trial % 11 == 2 && p.kv.n_segs > 0) p.kv.start[0] = cu.back() + 1;
    if (trial % 13 == 3) p.n_kv_heads = int32_t(uni(-2, 9));
    if (trial % 17 == 4) p.q_tok_stride = int32_t(uni(-16, 4096));
    if (trial % 19 == 5) p.n_docs = 0;
    if (trial % 23 == 6) cu[size_t(n_docs)] = cu[0] - 1;
    if (trial % 29 == 7) p.q.n_segs = HYDRA_MAX_SEGS + 1;
    if (trial % 31 == 8) p.n_heads = int32_t(uni(-1, 5000));
    hydra::Problem pr;
    if (hydra::check_problem(&p, &pr) != HYDRA_OK) {
      ++refused;
      continue;
    }
    std::vector<int32_t> items;
    hydra::plan_items(pr, 0, &items);
    hydra::plan_items(pr, 1, &items);
    const hydra::WsLayout w = hydra::ws_layout(pr);
    if (w.total < w.lse2_off) return 3;
    pairs += hydra::visible_pairs(pr);
    ++planned;
  }

  int64_t placed = 0, sched_refused = 0;
  for (int trial = 0; trial < 400; ++trial) {
    const int64_t n = uni(1, 300);
    std::vector<int64_t> len(static_cast<size_t>(n));
    for (auto& x : len) x = uni(1, 1 << 15);
    if (trial % 9 == 1) len[0] = 0;                 // malformed length
    hydra_sched_config_t cfg{};
    cfg.n_ranks = int32_t(1) << uni(0, 8);
    cfg.token_budget = uni(512, 1 << 16);
    cfg.pp = int32_t(uni(1, 8));
    cfg.theta_over_c = double(uni(0, 100)) / 10.0;
    cfg.cap = trial % 5 == 2 ? int32_t(1) << uni(0, 4) : 0;
    cfg.balance_ratio = trial % 3 == 0 ? double(uni(1, 10)) / 10.0 : 0.0;
    if (trial % 13 == 3) cfg.n_ranks = int32_t(uni(-1, 3));
    std::vector<int32_t> mb(static_cast<size_t>(n)), st(static_cast<size_t>(n)), sz(static_cast<size_t>(n));
    hydra_sched_summary_t sum{};
    if (hydra_schedule(len.data(), n, &cfg, mb.data(), st.data(), sz.data(), trial % 4 ? &sum : nullptr) == HYDRA_OK)
      ++placed;
    else
      ++sched_refused;
  }
  std::printf("planned %lld refused %lld pairs %lld scheduled %lld refused %lld\n", (long long)planned,
              (long long)refused, (long long)pairs, (long long)placed, (long long)sched_refused);
  return 0;
}
