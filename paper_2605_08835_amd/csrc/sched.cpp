// Host-side sequence planner of the inter-concurrency scheduler (Sec. III-D,
// Problem P and Alg. 1): a dynamic program over (UNet tasks done, VAE tasks
// done, Skip-CFG tasks used) with the lookup-table latencies tau(m, n, k) and
// delta(m, n, k) of the offline profiler (Sec. III-C).  No GPU work.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <string>
#include <vector>

#include "synerdiff_sched.h"

namespace sd {
extern thread_local std::string g_err;
}

namespace {

struct Label {
  double c, t;
  int prev_state, prev_label;  // -1 at the start
  int m, n, k;
};

}  // namespace

extern "C" sd_status synerdiff_plan_sequence(int32_t M, int32_t N, int32_t K, int32_t bmax, const double* tau,
                                             const double* delta, double T_lim, int32_t mode, int32_t max_stages,
                                             int32_t* seq, int32_t* n_stages, double* cost, double* time) {
  using sd::g_err;
  if (!tau || !delta || !n_stages || !cost || !time || (max_stages > 0 && !seq)) {
    g_err = "NULL argument";
    return SD_ERR_INVALID_ARG;
  }
  if (M < 0 || N < 0 || K < 0 || bmax < 1 || bmax > 64 || (mode != 0 && mode != 1) || max_stages < 0) {
    g_err = "need M, N, K >= 0, 1 <= bmax <= 64, mode 0 or 1";
    return SD_ERR_INVALID_ARG;
  }
  if ((long)(M + 1) * (N + 1) * (K + 1) > 50000000L) {
    g_err = "state space too large";
    return SD_ERR_UNSUPPORTED;
  }
  const int B = bmax + 1;
  auto at = [&](const double* t, int m, int n, int k) { return t[((size_t)m * B + n) * B + k]; };
  for (int m = 1; m <= bmax; ++m)
    for (int n = 0; n <= m; ++n)
      for (int k = 0; k <= m; ++k)
        if (!std::isfinite(at(tau, m, n, k)) || !std::isfinite(at(delta, m, n, k)) || at(tau, m, n, k) < 0) {
          g_err = "lookup table entries must be finite (tau >= 0)";
          return SD_ERR_INVALID_ARG;
        }
  const auto sid = [&](int i, int j, int u) { return (i * (N + 1) + j) * (K + 1) + u; };
  const int S = (M + 1) * (N + 1) * (K + 1);
  std::vector<std::vector<Label>> lab(S);
  lab[sid(0, 0, 0)].push_back(Label{0.0, 0.0, -1, -1, 0, 0, 0});
  // states in lexicographic order (every action has m >= 1, so i grows);
  // actions (m, n, k) in lexicographic order
  for (int i = 0; i <= M; ++i)
    for (int j = 0; j <= N; ++j)
      for (int u = 0; u <= K; ++u) {
        const int s = sid(i, j, u);
        for (int li = 0; li < (int)lab[s].size(); ++li) {
          const double c = lab[s][li].c, t = lab[s][li].t;
          for (int m = 1; m <= bmax && i + m <= M; ++m)
            for (int n = 0; n <= m && j + n <= N; ++n)
              for (int k = 0; k <= m && u + k <= K; ++k) {
                const double t_new = t + at(tau, m, n, k);
                if (t_new > T_lim) continue;
                const double cv = n > 0 ? t + at(delta, m, n, k) : 0.0;
                const double c_new = c + cv * n;
                std::vector<Label>& L = lab[sid(i + m, j + n, u + k)];
                const Label nl{c_new, t_new, s, li, m, n, k};
                if (mode == 0) {  // Alg. 1: one label, replaced by a strictly smaller cost
                  if (L.empty())
                    L.push_back(nl);
                  else if (c_new < L[0].c)
                    L[0] = nl;
                } else {  // non-dominated labels
                  bool dom = false;
                  for (const Label& o : L)
                    if (o.c <= c_new && o.t <= t_new) {
                      dom = true;
                      break;
                    }
                  if (dom) continue;
                  L.erase(std::remove_if(L.begin(), L.end(),
                                         [&](const Label& o) { return c_new <= o.c && t_new <= o.t; }),
                          L.end());
                  L.push_back(nl);
                }
              }
        }
      }
  int bs = -1, bl = -1;
  for (int u = 0; u <= K; ++u) {
    const int s = sid(M, N, u);
    for (int li = 0; li < (int)lab[s].size(); ++li) {
      const Label& x = lab[s][li];
      // Alg. 1: the first u with the smallest cost; exact: smallest (cost, time)
      if (bs < 0 || x.c < lab[bs][bl].c || (mode == 1 && x.c == lab[bs][bl].c && x.t < lab[bs][bl].t)) {
        bs = s;
        bl = li;
      }
    }
  }
  if (bs < 0) {
    *n_stages = 0;
    *cost = *time = INFINITY;
    g_err = "no sequence meets the throughput cap";
    return SD_ERR_UNSUPPORTED;
  }
  *cost = lab[bs][bl].c;
  *time = lab[bs][bl].t;
  std::vector<int> rev;
  for (int s = bs, l = bl; lab[s][l].prev_state >= 0;) {
    const Label& x = lab[s][l];
    rev.push_back(x.m);
    rev.push_back(x.n);
    rev.push_back(x.k);
    const int ps = x.prev_state, pl = x.prev_label;
    s = ps;
    l = pl;
  }
  const int ns = (int)rev.size() / 3;
  *n_stages = ns;
  if (ns > max_stages) {
    g_err = "the sequence has more stages than max_stages";
    return SD_ERR_CAPACITY;
  }
  for (int t = 0; t < ns; ++t)
    for (int e = 0; e < 3; ++e) seq[3 * t + e] = rev[3 * (ns - 1 - t) + e];
  return SD_OK;
}
