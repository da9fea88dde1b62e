// Host-code workout for AddressSanitizer / UndefinedBehaviorSanitizer builds
// (built and run by tests/test_sanitizers.py with g++ -fsanitize=address,
// undefined; no GPU code is involved).  It drives the library's synchronous
// host helpers (topology table, path validation, draft pruning and packing,
// tree-mask converter) and the C oracle over exhaustive small drafts, random
// drafts up to the size limits and malformed inputs, with every buffer sized
// exactly, and cross-checks the host topology against the oracle's.  Exit
// status 0 means every check held; the sanitizers abort on the first memory
// or undefined-behaviour error.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <random>
#include <vector>

#include "kernels.hpp"
#include "layer_ops.hpp"
#include "sla.h"

// The host helpers never launch; the launchers the rest of the library
// defines in its HIP sources are stubbed out so that no GPU code is built.
namespace sla {
hipError_t launch_verify_serial(const VerifyArgs &, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_verify_hybrid(const VerifyArgs &, int, hipStream_t) { return hipErrorInvalidValue; }
bool parallel_supported(int, int, int, int) { return false; }
hipError_t launch_verify_parallel(const VerifyArgs &, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_verify_decode(const VerifyArgs &, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_commit(const CommitArgs &, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_topology(const TopologyArgs &, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_conv(const ConvArgs &, int, bool, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_prune(const PruneArgs &, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_mask_to_parent(const MaskArgs &, hipStream_t) { return hipErrorInvalidValue; }
}  // namespace sla

extern "C" {
int oracle_topology(const int32_t *parent, int n, int32_t *depth, uint64_t *anc, int32_t *order,
                    int32_t *n_children, int32_t *max_depth);
int oracle_validate_path(const int32_t *parent, int n, const int32_t *path, int len);
int oracle_verify_family(int family, int B, int H, int dk, int dv, int n, const double *state, const double *q,
                         const double *k, const double *v, const double *gate, const double *beta,
                         const int32_t *parent, double *out, int32_t *status);
int oracle_commit_family(int family, int B, int H, int dk, int dv, int n, double *state, const double *k,
                         const double *v, const double *gate, const double *beta, const int32_t *parent,
                         const int32_t *path, int path_stride, const int32_t *len, int32_t *status);
int oracle_conv_verify(int B, int D, int K, int n, const double *conv_state, const double *x, const double *w,
                       const double *bias, int activation, const int32_t *parent, double *y, int32_t *status);
int oracle_conv_commit(int B, int D, int K, int n, double *conv_state, const double *x, const int32_t *parent,
                       const int32_t *path, int path_stride, const int32_t *len, int32_t *status);
}

static int failures = 0;
#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
      ++failures;                                                 \
    }                                                             \
  } while (0)

static std::mt19937_64 rng(12345);

static int uni(int lo, int hi) {  // inclusive
  return std::uniform_int_distribution<int>(lo, hi)(rng);
}

static std::vector<int32_t> random_parent(int n, bool valid) {
  std::vector<int32_t> p(n);
  for (int j = 0; j < n; ++j) p[j] = uni(-1, j - 1);
  if (!valid && n > 0) p[uni(0, n - 1)] = uni(0, 1) ? uni(n, n + 5) : uni(-7, -2);
  return p;
}

static void topology_case(const std::vector<int32_t> &p) {
  const int n = (int)p.size();
  std::vector<int32_t> d1(n), o1(n), c1(n), d2(n), o2(n), c2(n);
  std::vector<uint64_t> a1(n), a2(n);
  int32_t m1 = -1, m2 = -1;
  const int s1 = sla_topology_host(p.data(), n, d1.data(), a1.data(), o1.data(), c1.data(), &m1);
  const int s2 = oracle_topology(p.data(), n, d2.data(), a2.data(), o2.data(), c2.data(), &m2);
  CHECK((s1 == SLA_OK) == (s2 == 0));
  if (s1 == SLA_OK && s2 == 0) {
    CHECK(d1 == d2 && a1 == a2 && o1 == o2 && c1 == c2 && m1 == m2);
    // every root path is a valid accepted path; a broken one is not
    for (int j = 0; j < n; ++j) {
      std::vector<int32_t> path;
      for (int x = j; x != -1; x = p[x]) path.insert(path.begin(), x);
      CHECK(sla_validate_path_host(p.data(), n, path.data(), (int)path.size()) == SLA_OK);
      CHECK(oracle_validate_path(p.data(), n, path.data(), (int)path.size()) == 0);
      path.back() = (path.back() + 1) % (n + 1);
      const int v1 = sla_validate_path_host(p.data(), n, path.data(), (int)path.size());
      const int v2 = oracle_validate_path(p.data(), n, path.data(), (int)path.size());
      CHECK((v1 == SLA_OK) == (v2 == 0));
    }
    // tree mask -> parent array round trip
    std::vector<int32_t> back(n);
    CHECK(sla_tree_mask_to_parent_host(a1.data(), n, back.data()) == SLA_OK);
    CHECK(back == p);
    std::vector<uint64_t> bad = a1;
    bad[uni(0, n - 1)] ^= 1ull << uni(0, n - 1);
    sla_tree_mask_to_parent_host(bad.data(), n, back.data());  // either verdict; must stay in bounds
  }
}

static void prune_case(int n, double tau, int budget, bool corrupt) {
  std::vector<int32_t> p = random_parent(n, true), pp(n), im(n);
  std::vector<float> lp(n), sc(n);
  for (int j = 0; j < n; ++j) lp[j] = -std::uniform_real_distribution<float>(0.f, 4.f)(rng);
  if (corrupt) lp[uni(0, n - 1)] = uni(0, 1) ? 0.5f : NAN;
  int32_t count = -1;
  const int st = sla_prune_host(p.data(), lp.data(), n, (float)tau, budget, pp.data(), im.data(), &count, sc.data());
  if (corrupt) {
    CHECK(st == SLA_ERR_SCORE);
    return;
  }
  CHECK(st == SLA_OK);
  CHECK(count >= 1 && count <= n);
  if (budget > 0) CHECK(count <= budget);
  for (int j = 0; j < count; ++j) {
    CHECK(im[j] >= 0 && im[j] < n);
    CHECK(pp[j] >= -1 && pp[j] < j);
    if (j > 0) CHECK(im[j] > im[j - 1]);
  }
  for (int j = count; j < n; ++j) CHECK(pp[j] == -1 && im[j] == -1);
  if (count <= SLA_MAX_NODES) topology_case(std::vector<int32_t>(pp.begin(), pp.begin() + count));
}

static void oracle_case(int family, int B, int H, int dk, int dv, int n) {
  const size_t bnh = (size_t)B * n * H, gw = family == 3 ? (size_t)dk : 1;
  std::vector<double> S((size_t)B * H * dk * dv), q(bnh * dk), k(bnh * dk), v(bnh * dv), g(bnh * gw), be(bnh),
      out(bnh * dv);
  std::normal_distribution<double> N(0.0, 1.0);
  for (auto &x : S) x = 0.02 * N(rng);
  for (auto &x : q) x = N(rng) / sqrt((double)dk);
  for (auto &x : k) x = N(rng) / sqrt((double)dk);
  for (auto &x : v) x = N(rng);
  for (auto &x : g) x = std::uniform_real_distribution<double>(0.5, 1.0)(rng);
  for (auto &x : be) x = std::uniform_real_distribution<double>(0.0, 1.0)(rng);
  std::vector<int32_t> par((size_t)B * n), path((size_t)B * n, -1), len(B), st(B);
  for (int b = 0; b < B; ++b) {
    std::vector<int32_t> p = random_parent(n, b != 1 || B < 3);  // sequence 1 malformed when B >= 3
    memcpy(&par[(size_t)b * n], p.data(), sizeof(int32_t) * n);
    int L = 0;
    {
      std::vector<int32_t> pth;
      bool ok = true;
      for (int x = uni(0, n - 1); x != -1; x = p[x]) {
        if (x < -1 || x >= n || pth.size() > (size_t)n) {
          ok = false;
          break;
        }
        pth.insert(pth.begin(), x);
      }
      if (ok) {
        L = (int)pth.size();
        memcpy(&path[(size_t)b * n], pth.data(), sizeof(int32_t) * L);
      }
    }
    len[b] = L;
  }
  const double *gp = family == 1 ? nullptr : g.data();
  const double *bp = (family == 0 || family == 1) ? be.data() : nullptr;
  oracle_verify_family(family, B, H, dk, dv, n, S.data(), q.data(), k.data(), v.data(), gp, bp, par.data(),
                       out.data(), st.data());
  oracle_commit_family(family, B, H, dk, dv, n, S.data(), k.data(), v.data(), gp, bp, par.data(), path.data(), n,
                       len.data(), st.data());
  // the short convolution on the same drafts
  const int D = 8 * uni(1, 4), K = uni(1, 4);
  std::vector<double> C((size_t)B * (K - 1) * D + 1), x((size_t)B * n * D), w((size_t)D * K), bias(D),
      y((size_t)B * n * D);
  for (auto &z : x) z = N(rng);
  for (auto &z : C) z = N(rng);
  for (auto &z : w) z = N(rng);
  for (auto &z : bias) z = N(rng);
  oracle_conv_verify(B, D, K, n, C.data(), x.data(), w.data(), bias.data(), 1, par.data(), y.data(), st.data());
  oracle_conv_commit(B, D, K, n, C.data(), x.data(), par.data(), path.data(), n, len.data(), st.data());
}

int main() {
  // exhaustive small drafts: every parent array with parent[j] in [-1, j)
  for (int n = 1; n <= 6; ++n) {
    std::vector<int32_t> p(n, -1);
    while (true) {
      topology_case(p);
      int j = n - 1;
      while (j >= 0 && p[j] == j - 1) p[j--] = -1;
      if (j < 0) break;
      ++p[j];
    }
  }
  // random drafts up to the node limit, valid and malformed
  for (int it = 0; it < 3000; ++it) {
    const int n = uni(1, SLA_MAX_NODES);
    topology_case(random_parent(n, it % 5 != 0));
  }
  // size limits and null pointers return an error without touching memory
  {
    int32_t p[1] = {-1}, d[1], o[1], c[1], md;
    uint64_t a[1];
    CHECK(sla_topology_host(p, 0, d, a, o, c, &md) == SLA_ERR_SHAPE);
    CHECK(sla_topology_host(p, SLA_MAX_NODES + 1, d, a, o, c, &md) == SLA_ERR_SHAPE);
    CHECK(sla_topology_host(nullptr, 1, d, a, o, c, &md) == SLA_ERR_NULL);
    CHECK(sla_validate_path_host(p, 1, nullptr, 0) == SLA_OK);
    CHECK(sla_validate_path_host(p, 1, nullptr, 1) == SLA_ERR_NULL);
    CHECK(sla_tree_mask_to_parent_host(a, 0, o) == SLA_ERR_SHAPE);
    float lp[1] = {-1.f};
    int32_t cnt;
    CHECK(sla_prune_host(p, lp, 0, 1.f, 0, d, o, &cnt, nullptr) == SLA_ERR_SHAPE);
    CHECK(sla_prune_host(p, lp, 1, -1.f, 0, d, o, &cnt, nullptr) == SLA_ERR_SHAPE);
    CHECK(sla_prune_host(nullptr, lp, 1, 1.f, 0, d, o, &cnt, nullptr) == SLA_ERR_NULL);
    CHECK(sla_factors_bytes(nullptr) == 0);
    CHECK(strlen(sla_status_string(-100)) > 0);
  }
  // pruning: sizes past the device limit, every budget regime, bad scores
  for (int it = 0; it < 600; ++it) {
    const int n = it % 3 == 0 ? uni(65, 700) : uni(1, 64);
    const double tau = uni(0, 3) == 0 ? INFINITY : std::uniform_real_distribution<double>(0.0, 6.0)(rng);
    prune_case(n, tau, uni(-2, n + 2), it % 17 == 0);
  }
  // the oracle on small shapes, every family, with a malformed sequence
  for (int it = 0; it < 60; ++it)
    oracle_case(it % 4, uni(1, 4), uni(1, 3), 4 * uni(1, 4), 4 * uni(1, 4), uni(1, 12));
  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("sanitized host checks passed\n");
  return 0;
}
