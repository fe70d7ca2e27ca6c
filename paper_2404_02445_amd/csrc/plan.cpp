// Hybrid partitioning (HyPAD, Sec. III-C, Algorithm 1) on a chain of planning
// nodes, and the sub-slice ranges of the horizontal strategy.  Host-only.
//
// Readings of the paper used here (the printed algorithm's indices are
// garbled):
//   * node elimination compares the original footprints of adjacent nodes,
//     |M_j - M_{j+1}| / M_j <= tau forbids the cut between them; merging never
//     changes a node's own footprint, so one pass is the fixpoint; edge
//     elimination is the identity on a chain of single-in/single-out nodes;
//   * the compute cost of a slice i..j is c_m * (max M * sum t) (Eq. 6 with
//     the slice sized for its peak layer); its communication cost is
//     c_n * (out_bytes_j / ratio_j) / bw, zero after the last node;
//   * DP over split points, i ascending with a strict '<' (ties keep the
//     longest last slice); with a fixed slice count the same recurrence runs
//     over (slices, node); the backtrack follows the stored argmin;
//   * parallelism: per slice, eta in 1..eta_max (k_max, and floor(M_g/lambda)
//     when lambda > 0) minimising sum (t_p + t_a) of Eq. 5 (ties: smallest eta),
//     assigned to the slice's RD nodes;
//   * the latency constraint of Eq. 6 is evaluated and reported, not enforced;
//   * the Uniform variant of the evaluation keeps the slice count and gives every
//     slice the same number of nodes (array_split sizes).
// Sums run in ascending node order so the doubles are reproducible.
#include <cmath>
#include <limits>
#include <vector>

#include "internal.h"

namespace mopar {
namespace {

constexpr double kInf = std::numeric_limits<double>::infinity();

struct Ctx {
    const mopar_layer_profile* L;
    int n;
    const mopar_plan_opts* o;
};

double cost_cal(const Ctx& c, int i, int j) {   // 1-based inclusive
    double mx = 0.0, st = 0.0;
    for (int l = i; l <= j; ++l) {
        mx = std::fmax(mx, c.L[l - 1].mem_bytes);
        st = st + c.L[l - 1].time_s;
    }
    return c.o->c_m * (mx * st);
}

double t_comm(const Ctx& c, int j) {             // boundary after node j (1-based, j < n)
    const double r = c.o->ratio ? c.o->ratio[j - 1] : 1.0;
    return (c.L[j - 1].out_bytes / r) / c.o->bw_Bps;
}

double cost_com(const Ctx& c, int j) { return j == c.n ? 0.0 : c.o->c_n * t_comm(c, j); }

}  // namespace

int plan_slices_impl(const mopar_layer_profile* L, int32_t n, const mopar_plan_opts* o, mopar_plan* out) {
    if (!L || !o || !out) return set_error(MOPAR_E_ARG, "mopar_plan_slices: null argument");
    if (n < 1) return set_error(MOPAR_E_ARG, "mopar_plan_slices: n must be >= 1");
    if (!out->slice_end || !out->k) return set_error(MOPAR_E_ARG, "mopar_plan_slices: plan arrays are null");
    if (out->n_layers < n) return set_error(MOPAR_E_ARG, "mopar_plan_slices: plan capacity n_layers < n");
    if (!(o->bw_Bps > 0.0)) return set_error(MOPAR_E_ARG, "mopar_plan_slices: bw_Bps must be > 0");
    for (int l = 0; l < n; ++l)
        if (!(L[l].mem_bytes > 0.0) || !(L[l].time_s >= 0.0) || !(L[l].out_bytes >= 0.0) || L[l].rd_width < 0)
            return set_error(MOPAR_E_ARG, "mopar_plan_slices: layer profile " + std::to_string(l) +
                                              " needs mem_bytes > 0, time_s >= 0, out_bytes >= 0, rd_width >= 0");
    if (o->ratio)
        for (int j = 0; j + 1 < n; ++j)
            if (!(o->ratio[j] > 0.0)) return set_error(MOPAR_E_ARG, "mopar_plan_slices: ratios must be > 0");
    const int kmax = o->k_max < 1 ? 1 : o->k_max;
    if (o->k_override)
        for (int l = 0; l < n; ++l) {
            const int k = o->k_override[l];
            if (k < 0 || (k > 0 && (L[l].rd_width == 0 ? k > 1 : k > L[l].rd_width)))
                return set_error(MOPAR_E_ARG, "mopar_plan_slices: k_override[" + std::to_string(l) +
                                                  "] needs an RD op at least that wide");
            // measured tables hold t_p / t_a for eta = 1 .. k_max only
            if (k > kmax && (o->tp_table || o->ta_table))
                return set_error(MOPAR_E_ARG, "mopar_plan_slices: k_override[" + std::to_string(l) +
                                                  "] exceeds k_max, beyond the measured tables");
        }

    // step 1: graph simplification
    std::vector<int> allowed(n > 1 ? n - 1 : 0, 1);
    if (o->allowed_cut) {
        for (int j = 0; j + 1 < n; ++j) allowed[j] = o->allowed_cut[j] ? 1 : 0;
    } else if (o->elim_tau >= 0.0) {
        for (int j = 0; j + 1 < n; ++j)
            allowed[j] = (std::fabs(L[j].mem_bytes - L[j + 1].mem_bytes) / L[j].mem_bytes <= o->elim_tau) ? 0 : 1;
    }
    auto cut_ok = [&](int i) { return i == 1 || allowed[i - 2] == 1; };

    // step 2: DP over split points and backtrack
    const Ctx c{L, n, o};
    const int K = o->n_slices;
    if (K < 0 || K > n) return set_error(MOPAR_E_INFEASIBLE, "mopar_plan_slices: n_slices out of range");
    std::vector<int> ends;
    double cost;
    if (o->uniform) {
        // Uniform: K slices of equal node counts (the first n mod K one longer)
        if (K == 0) return set_error(MOPAR_E_ARG, "mopar_plan_slices: the uniform variant needs n_slices > 0");
        const int q = n / K, r = n % K;
        std::vector<int> fwd;
        for (int s = 0, e = -1; s < K; ++s) {
            e += q + (s < r ? 1 : 0);
            fwd.push_back(e);
        }
        cost = 0.0;
        for (int s = 0, i = 1; s < K; ++s) {
            const int j = fwd[s] + 1;
            cost = cost + (cost_cal(c, i, j) + cost_com(c, j));
            i = j + 1;
        }
        ends.assign(fwd.rbegin(), fwd.rend());
    } else if (K == 0) {
        std::vector<double> dp(n + 1, kInf);
        std::vector<int> arg(n + 1, 0);
        dp[0] = 0.0;
        for (int j = 1; j <= n; ++j)
            for (int i = 1; i <= j; ++i) {
                if (!cut_ok(i) || dp[i - 1] == kInf) continue;
                const double v = dp[i - 1] + (cost_cal(c, i, j) + cost_com(c, j));
                if (v < dp[j]) {
                    dp[j] = v;
                    arg[j] = i;
                }
            }
        for (int j = n; j > 0; j = arg[j] - 1) ends.push_back(j - 1);
        cost = dp[n];
    } else {
        std::vector<double> dp((K + 1) * (n + 1), kInf);
        std::vector<int> arg((K + 1) * (n + 1), 0);
        auto D = [&](int s, int j) -> double& { return dp[s * (n + 1) + j]; };
        auto A = [&](int s, int j) -> int& { return arg[s * (n + 1) + j]; };
        D(0, 0) = 0.0;
        for (int s = 1; s <= K; ++s)
            for (int j = s; j <= n; ++j)
                for (int i = s; i <= j; ++i) {
                    if ((s == 1) != (i == 1)) continue;
                    if (!cut_ok(i) || D(s - 1, i - 1) == kInf) continue;
                    const double v = D(s - 1, i - 1) + (cost_cal(c, i, j) + cost_com(c, j));
                    if (v < D(s, j)) {
                        D(s, j) = v;
                        A(s, j) = i;
                    }
                }
        if (D(K, n) == kInf)
            return set_error(MOPAR_E_INFEASIBLE, "mopar_plan_slices: fewer admissible cuts than n_slices - 1");
        for (int j = n, s = K; j > 0; --s) {
            ends.push_back(j - 1);
            j = A(s, j) - 1;
        }
        cost = D(K, n);
    }
    std::vector<int> e(ends.rbegin(), ends.rend());

    // step 3: parallelism per slice
    auto tp = [&](int l, int eta) { return o->tp_table ? o->tp_table[l * kmax + eta - 1] : L[l].time_s; };
    auto ta = [&](int l, int eta) { return o->ta_table ? o->ta_table[l * kmax + eta - 1] : 0.0; };
    std::vector<int> k(n, 1);
    int start = 0;
    for (int end : e) {
        double mg = 0.0;
        for (int l = start; l <= end; ++l) mg = std::fmax(mg, L[l].mem_bytes);
        int emax = kmax;
        if (o->lambda_bytes > 0.0) {
            const double cap = std::floor(mg / o->lambda_bytes);
            if (cap < emax) emax = static_cast<int>(cap);
        }
        if (emax < 1) emax = 1;
        double best = kInf;
        int best_e = 1;
        for (int eta = 1; eta <= emax; ++eta) {
            double tot = 0.0;
            for (int l = start; l <= end; ++l) {
                const int ee = L[l].rd_width > 0 ? eta : 1;
                tot = tot + (tp(l, ee) + ta(l, ee));
            }
            if (tot < best) {
                best = tot;
                best_e = eta;
            }
        }
        for (int l = start; l <= end; ++l)
            if (L[l].rd_width > 0) k[l] = best_e < L[l].rd_width ? best_e : L[l].rd_width;
        start = end + 1;
    }
    if (o->k_override)
        for (int l = 0; l < n; ++l)
            if (o->k_override[l] > 0) k[l] = o->k_override[l];

    // latency (Eq. 5) and the unsplit reference
    double t_tau = 0.0;
    for (int l = 0; l < n; ++l) t_tau = t_tau + (tp(l, k[l]) + ta(l, k[l]));
    for (size_t s = 0; s + 1 < e.size(); ++s) t_tau = t_tau + t_comm(c, e[s] + 1);
    double t_un = 0.0;
    for (int l = 0; l < n; ++l) t_un = t_un + L[l].time_s;

    out->n_slices = static_cast<int32_t>(e.size());
    for (size_t s = 0; s < e.size(); ++s) out->slice_end[s] = e[s];
    for (int l = 0; l < n; ++l) out->k[l] = k[l];
    out->cost = cost;
    out->t_tau = t_tau;
    out->t_unsplit = t_un;
    out->latency_ok = t_tau <= t_un ? 1 : 0;
    return MOPAR_OK;
}

int subslice_range_impl(int32_t n, int32_t k, int32_t j, int32_t* lo, int32_t* hi) {
    if (!lo || !hi) return set_error(MOPAR_E_ARG, "mopar_subslice_range: null output");
    if (!(k >= 1 && k <= n && j >= 0 && j < k))
        return set_error(MOPAR_E_ARG, "mopar_subslice_range: need 1 <= k <= n and 0 <= j < k");
    const int32_t q = n / k, r = n % k;
    *lo = j * q + (j < r ? j : r);
    *hi = (j + 1) * q + (j + 1 < r ? j + 1 : r);
    return MOPAR_OK;
}

}  // namespace mopar
