// Prompt-routing control plane of an Argus cluster, on the host (no GPU work):
// the Optimized Distribution Aligner that builds the Probabilistic Approximation
// Shift Map from the classifier's demand histogram and the solver's load split
// (Sec. 4.3, Alg. 1), the scheduler's draw from that map and the greedy worker
// selector of Eq. 3 (Sec. 4.4). Levels are indexed from the slowest / most accurate
// (0) to the fastest / most approximate (n - 1).
#include <cmath>
#include <vector>

#include "model.h"

namespace dn {

// One sweep from the fastest level to the slowest. `own[k]` is what is left of level
// k's own prompts (levels not yet visited hold nothing else); `carry[o]` is the mass
// of origin o travelling left from the level just visited. At level i the mass present
// is own[i] plus the carry: if it exceeds F[i], the fraction F[i] / present is served
// at i and the rest of every origin's share travels on to i - 1 (a step to a slower
// level loses no quality); otherwise everything present is served at i and the
// shortfall is taken from the nearest slower levels' own prompts, nearest first.
// served[o * n + j]: mass of origin o served at level j.
void oda_pasm(const double* H, const double* F, int n, double* T) {
  std::vector<double> own(H, H + n), carry(n, 0.0), served((size_t)n * n, 0.0);
  for (int i = n - 1; i >= 0; --i) {
    double present = own[i];
    for (int o = i + 1; o < n; ++o) present += carry[o];
    if (present > F[i] && i > 0) {
      const double stay = F[i] / present;
      served[(size_t)i * n + i] += own[i] * stay;
      carry[i] = own[i] - own[i] * stay;
      for (int o = i + 1; o < n; ++o) {
        const double s = carry[o] * stay;
        served[(size_t)o * n + i] += s;
        carry[o] -= s;
      }
      own[i] = 0.0;
    } else {
      served[(size_t)i * n + i] += own[i];
      for (int o = i + 1; o < n; ++o) {
        served[(size_t)o * n + i] += carry[o];
        carry[o] = 0.0;
      }
      own[i] = 0.0;
      double need = F[i] - present;
      for (int k = i - 1; k >= 0 && need > 0.0; --k) {
        const double take = own[k] < need ? own[k] : need;
        served[(size_t)k * n + i] += take;
        own[k] -= take;
        need -= take;
      }
    }
  }
  for (int o = 0; o < n; ++o)
    for (int j = 0; j < n; ++j)
      T[(size_t)o * n + j] = H[o] > 0.0 ? served[(size_t)o * n + j] / H[o] : (o == j ? 1.0 : 0.0);
}

}  // namespace dn

namespace {

thread_local std::string g_ctl_error;

template <typename Fn> dn_status ctl_guarded(Fn&& f) {
  try {
    g_ctl_error.clear();
    f();
    return DN_OK;
  } catch (const dn::Error& e) {
    g_ctl_error = e.what();
    return static_cast<dn_status>(e.code);
  } catch (const std::bad_alloc&) {
    g_ctl_error = "host allocation failed";
    return DN_ENOMEM;
  } catch (...) {
    g_ctl_error = "unknown error";
    return DN_EINVAL;
  }
}

}  // namespace

extern "C" {

dn_status argus_oda(const double* H, const double* F, int32_t n, double* pasm) {
  return ctl_guarded([&] {
    DN_CHECK(H && F && pasm, "argus_oda: null pointer");
    DN_CHECK(n >= 1 && n <= ARGUS_MAX_LEVELS, "argus_oda: n must be in [1, 64]");
    double sh = 0.0, sf = 0.0;
    for (int i = 0; i < n; ++i) {
      DN_CHECK(std::isfinite(H[i]) && std::isfinite(F[i]) && H[i] >= 0.0 && F[i] >= 0.0,
               "argus_oda: histograms must be finite and non-negative");
      sh += H[i];
      sf += F[i];
    }
    DN_CHECK(sh > 0.0, "argus_oda: empty demand histogram");
    DN_CHECK(std::fabs(sh - sf) <= 1e-9 * (sh > 1.0 ? sh : 1.0), "argus_oda: H and F must have the same total");
    dn::oda_pasm(H, F, n, pasm);
  });
}

dn_status argus_route(const double* pasm, int32_t n, int32_t level, double u, int32_t* out_level) {
  return ctl_guarded([&] {
    DN_CHECK(pasm && out_level, "argus_route: null pointer");
    DN_CHECK(n >= 1 && n <= ARGUS_MAX_LEVELS, "argus_route: n must be in [1, 64]");
    DN_CHECK(level >= 0 && level < n, "argus_route: level out of range");
    DN_CHECK(u >= 0.0 && u < 1.0, "argus_route: u must be in [0, 1)");
    const double* row = pasm + (size_t)level * n;
    double c = 0.0;
    int last = level;
    for (int j = 0; j < n; ++j) {
      DN_CHECK(std::isfinite(row[j]) && row[j] >= 0.0, "argus_route: PASM row must be finite and non-negative");
      if (row[j] > 0.0) last = j;
    }
    for (int j = 0; j < n; ++j) {
      c += row[j];
      if (u < c) {
        *out_level = j;
        return;
      }
    }
    *out_level = last;
  });
}

dn_status argus_select_worker(const int32_t* queue_len, const double* t_proc, const int32_t* worker_level,
                              int32_t n_workers, int32_t level, int32_t* out_worker) {
  return ctl_guarded([&] {
    DN_CHECK(queue_len && t_proc && worker_level && out_worker, "argus_select_worker: null pointer");
    DN_CHECK(n_workers >= 1, "argus_select_worker: n_workers must be >= 1");
    int best = -1;
    double best_cost = 0.0;
    for (int w = 0; w < n_workers; ++w) {
      DN_CHECK(queue_len[w] >= 0 && std::isfinite(t_proc[w]) && t_proc[w] >= 0.0,
               "argus_select_worker: queue lengths and times must be non-negative");
      if (worker_level[w] != level) continue;
      const double cost = (double)queue_len[w] * t_proc[w];
      if (best < 0 || cost < best_cost) {
        best = w;
        best_cost = cost;
      }
    }
    *out_worker = best;
  });
}

const char* argus_last_error(void) { return g_ctl_error.c_str(); }

}  // extern "C"
