// CPU setup step of libstepq (offline, host memory only): the dual-axis
// scale fit of the initial states, the lifetime-ranked bit allocation, and
// the calibration side -- row-impact factors, candidate-format distortions,
// lifetime weights, the two allocators and the FP16 pivot choice.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <numeric>
#include <string>
#include <mutex>
#include <thread>
#include <vector>

#include "stepq.h"

namespace {

void fit_tiles(int64_t t0, int64_t t1, int32_t dk, int32_t dv, const float *S, const float *w, const uint8_t *bits,
               int levels, float *r, float *c)
{
    const double fl = std::ldexp(1.0, -60);
    std::vector<double> rd(dk);
    std::vector<double> cmax(dv);
    for (int64_t t = t0; t < t1; ++t) {
        const float *St = S + t * dk * static_cast<int64_t>(dv);
        for (int i = 0; i < dk; ++i) {
            double m = 0.0;
            const float *row = St + static_cast<int64_t>(i) * dv;
            for (int j = 0; j < dv; ++j) m += std::fabs(static_cast<double>(row[j]));
            m /= static_cast<double>(dv);
            const double wi = w ? static_cast<double>(w[t * dk + i]) : 1.0;
            double ri = std::sqrt(m / wi);
            if (ri < fl) ri = fl;
            const float rf = static_cast<float>(ri);
            r[t * dk + i] = rf;
            rd[i] = static_cast<double>(rf);
        }
        std::fill(cmax.begin(), cmax.end(), 0.0);
        for (int i = 0; i < dk; ++i) {
            if (bits && bits[t * dk + i] == 16) continue;    // pivot rows keep their own values
            const float *row = St + static_cast<int64_t>(i) * dv;
            const double inv = rd[i];
            double top = 1.0;                        // the width's top level: 1 (N1), 2^(8-b) q_b (N2)
            if (levels == STEPQ_LEVELS_POW2) {
                const int b = bits[t * dk + i];
                top = static_cast<double>((1 << (b - 1)) - 1) * std::ldexp(1.0, 8 - b);
            }
            for (int j = 0; j < dv; ++j) {
                double a = std::fabs(static_cast<double>(row[j])) / inv;
                if (levels == STEPQ_LEVELS_POW2) a /= top;
                if (a > cmax[j]) cmax[j] = a;
            }
        }
        for (int j = 0; j < dv; ++j) {
            double cj = cmax[j] < fl ? fl : cmax[j];
            float cf = static_cast<float>(cj);
            if (static_cast<double>(cf) < cj) cf = std::nextafter(cf, INFINITY);
            c[t * dv + j] = cf;
        }
    }
}

// ---- calibration helpers

double qb_of(int b) { return static_cast<double>((1 << (b - 1)) - 1); }

// The binary16 value nearest x (ties to even), as a double: round to 11
// significant bits, or to the subnormal spacing 2^-24, saturating to
// infinity from 65520 (half an ulp above the largest finite value) up.
double half_round(double x)
{
    if (!std::isfinite(x)) return x;
    const double a = std::fabs(x);
    if (a >= 65520.0) return std::copysign(std::numeric_limits<double>::infinity(), x);
    int e = 0;
    std::frexp(a, &e);                      // a = m 2^e, m in [0.5, 1)
    const int q = std::max(e - 11, -24);    // exponent of the spacing
    return std::copysign(std::ldexp(std::nearbyint(std::ldexp(a, -q)), q), x);
}

// The dual-axis fit of one state X [dk][dv] with widths b (16 = pivot row,
// left out) and factors w; writes the reconstruction R.  Follows Section 4.3
// and Appendix C.1 with the absmax start; scales stored as fp32.
void codec_tile(int dk, int dv, const double *X, const uint8_t *b, const double *w, double *R,
                std::vector<double> &r, std::vector<double> &c)
{
    const double fl = std::ldexp(1.0, -60);
    r.assign(dk, 1.0);
    c.assign(dv, 1.0);
    for (int i = 0; i < dk; ++i) {
        if (b[i] == 16) continue;
        double m = 0.0;
        for (int j = 0; j < dv; ++j) m += std::fabs(X[static_cast<size_t>(i) * dv + j]);
        m /= static_cast<double>(dv);
        double ri = std::sqrt(m / (w ? w[i] : 1.0));
        if (ri < fl) ri = fl;
        r[i] = static_cast<double>(static_cast<float>(ri));
    }
    for (int j = 0; j < dv; ++j) {
        double c0 = 0.0;
        for (int i = 0; i < dk; ++i) {
            if (b[i] == 16) continue;
            const double a = std::fabs(X[static_cast<size_t>(i) * dv + j]) / r[i];
            if (a > c0) c0 = a;
        }
        if (c0 < fl) c0 = fl;
        double num = 0.0, den = 0.0;
        for (int i = 0; i < dk; ++i) {
            if (b[i] == 16) continue;
            const double qb = qb_of(b[i]);
            double z = std::nearbyint(X[static_cast<size_t>(i) * dv + j] * qb / (r[i] * c0));
            z = std::min(qb, std::max(-qb, z));
            const double wi = w ? w[i] : 1.0;
            const double v = r[i] * z / qb;
            num += wi * wi * v * X[static_cast<size_t>(i) * dv + j];
            den += wi * wi * v * v;
        }
        double cj = den > 0.0 ? num / den : c0;
        if (cj < fl) cj = fl;
        c[j] = static_cast<double>(static_cast<float>(cj));
    }
    for (int i = 0; i < dk; ++i)
        for (int j = 0; j < dv; ++j) {
            const size_t e = static_cast<size_t>(i) * dv + j;
            if (b[i] == 16) {
                R[e] = half_round(X[e]);
                continue;
            }
            const double qb = qb_of(b[i]);
            double z = std::nearbyint(X[e] * qb / (r[i] * c[j]));
            z = std::min(qb, std::max(-qb, z));
            R[e] = r[i] * c[j] * z / qb;
        }
}

template <class F>
void parallel_for(int64_t n, int32_t n_threads, F &&f)
{
    int nt = n_threads > 0 ? n_threads : static_cast<int>(std::max(1u, std::thread::hardware_concurrency()));
    nt = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(nt, n)));
    if (nt == 1) {
        f(0, n);
        return;
    }
    std::vector<std::thread> pool;
    const int64_t per = (n + nt - 1) / nt;
    for (int k = 0; k < nt; ++k) {
        const int64_t a = k * per, b = std::min<int64_t>(n, a + per);
        if (a < b) pool.emplace_back(f, a, b);
    }
    for (auto &th : pool) th.join();
}

}  // namespace

extern "C" {

stepq_status stepq_setup_fit(int64_t n_tiles, int32_t d_k, int32_t d_v, const float *state, const float *row_weight,
                             float *r, float *c, int32_t n_threads)
{
    return stepq_setup_fit_ex(n_tiles, d_k, d_v, state, row_weight, nullptr, r, c, n_threads);
}

stepq_status stepq_setup_fit_ex(int64_t n_tiles, int32_t d_k, int32_t d_v, const float *state,
                                const float *row_weight, const uint8_t *row_bits, float *r, float *c,
                                int32_t n_threads)
{
    return stepq_setup_fit_levels(n_tiles, d_k, d_v, state, row_weight, row_bits, STEPQ_LEVELS_ABSMAX, r, c,
                                  n_threads);
}

stepq_status stepq_setup_fit_levels(int64_t n_tiles, int32_t d_k, int32_t d_v, const float *state,
                                    const float *row_weight, const uint8_t *row_bits, int32_t levels, float *r,
                                    float *c, int32_t n_threads)
{
    if (n_tiles < 0 || d_k < 1 || d_v < 1) return STEPQ_E_INVALID;
    if (levels != STEPQ_LEVELS_ABSMAX && levels != STEPQ_LEVELS_POW2) return STEPQ_E_INVALID;
    if (levels == STEPQ_LEVELS_POW2 && n_tiles > 0 && !row_bits) return STEPQ_E_INVALID;
    if (row_bits)
        for (int64_t e = 0; e < n_tiles * d_k; ++e)
            if (row_bits[e] != 2 && row_bits[e] != 4 && row_bits[e] != 8 && row_bits[e] != 16) return STEPQ_E_INVALID;
    if (n_tiles == 0) return STEPQ_OK;
    if (!state || !r || !c) return STEPQ_E_INVALID;
    int nt = n_threads > 0 ? n_threads : static_cast<int>(std::max(1u, std::thread::hardware_concurrency()));
    nt = static_cast<int>(std::min<int64_t>(nt, n_tiles));
    if (nt <= 1) {
        fit_tiles(0, n_tiles, d_k, d_v, state, row_weight, row_bits, levels, r, c);
        return STEPQ_OK;
    }
    std::vector<std::thread> pool;
    const int64_t per = (n_tiles + nt - 1) / nt;
    for (int k = 0; k < nt; ++k) {
        const int64_t t0 = k * per, t1 = std::min<int64_t>(n_tiles, t0 + per);
        if (t0 >= t1) break;
        pool.emplace_back(fit_tiles, t0, t1, d_k, d_v, state, row_weight, row_bits, levels, r, c);
    }
    for (auto &th : pool) th.join();
    return STEPQ_OK;
}

stepq_status stepq_setup_lifetime_bits(const double *gates, int32_t T, int32_t B, int32_t H, int32_t d_k,
                                       double budget, int32_t lo, int32_t hi, uint8_t *row_bits)
{
    if (!gates || !row_bits || T < 1 || B < 1 || H < 1 || d_k < 1) return STEPQ_E_INVALID;
    if (!(lo < hi) || budget < lo || budget > hi) return STEPQ_E_INVALID;
    for (int32_t wdt : {lo, hi})
        if (wdt != 2 && wdt != 4 && wdt != 8) return STEPQ_E_INVALID;
    // mean log retention per head over all calibration steps and requests
    std::vector<double> ell(H, 0.0);
    for (int32_t t = 0; t < T; ++t)
        for (int32_t b = 0; b < B; ++b)
            for (int32_t h = 0; h < H; ++h) {
                const double g = gates[(static_cast<int64_t>(t) * B + b) * H + h];
                if (!(g > 0.0)) return STEPQ_E_INVALID;
                ell[h] += std::log(g);
            }
    for (double &e : ell) e /= static_cast<double>(T) * B;
    // rows ranked by (l desc, head asc, row asc); the widest budget-share first
    std::vector<int32_t> order(static_cast<size_t>(H) * d_k);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
        const int32_t ha = a / d_k, hb = b / d_k;
        if (ell[ha] != ell[hb]) return ell[ha] > ell[hb];
        return a < b;
    });
    const int64_t n = static_cast<int64_t>(H) * d_k;
    const int64_t n_hi = static_cast<int64_t>(std::floor(n * (budget - lo) / (hi - lo) + 1e-9));
    for (int64_t u = 0; u < n; ++u) row_bits[order[u]] = static_cast<uint8_t>(u < n_hi ? hi : lo);
    return STEPQ_OK;
}

stepq_status stepq_setup_row_impact(int64_t T, int32_t H, int32_t d_k, const float *q, const float *k,
                                    const float *beta, const float *gate, int32_t gate_per_row, double gamma,
                                    float *row_weight, double *omega_out)
{
    if (T < 1 || H < 1 || d_k < 1 || !q || !k || !beta || !gate || !row_weight || !(gamma > 0.0))
        return STEPQ_E_INVALID;
    std::vector<double> omega(static_cast<size_t>(H) * d_k, 0.0);
    for (int64_t t = 0; t < T; ++t)
        for (int32_t h = 0; h < H; ++h) {
            const size_t base = (static_cast<size_t>(t) * H + h) * d_k;
            double kq = 0.0;
            for (int32_t i = 0; i < d_k; ++i) kq += static_cast<double>(k[base + i]) * static_cast<double>(q[base + i]);
            const double bt = beta[static_cast<size_t>(t) * H + h];
            for (int32_t i = 0; i < d_k; ++i) {
                const double d = gate_per_row ? static_cast<double>(gate[base + i])
                                              : static_cast<double>(gate[static_cast<size_t>(t) * H + h]);
                // (A^T q)_i with A = (I - beta k k^T) D
                const double g = d * (static_cast<double>(q[base + i]) - bt * static_cast<double>(k[base + i]) * kq);
                omega[static_cast<size_t>(h) * d_k + i] += g * g;
            }
        }
    const double fl = std::ldexp(1.0, -120);
    for (int32_t h = 0; h < H; ++h) {
        double lsum = 0.0;
        std::vector<double> p(d_k);
        for (int32_t i = 0; i < d_k; ++i) {
            double &om = omega[static_cast<size_t>(h) * d_k + i];
            om /= static_cast<double>(T);
            if (om < fl) om = fl;
            p[i] = std::pow(om, gamma / 2.0);
            lsum += std::log(p[i]);
        }
        const double gm = std::exp(lsum / d_k);
        for (int32_t i = 0; i < d_k; ++i) {
            row_weight[static_cast<size_t>(h) * d_k + i] = static_cast<float>(p[i] / gm);
            if (omega_out) omega_out[static_cast<size_t>(h) * d_k + i] = omega[static_cast<size_t>(h) * d_k + i];
        }
    }
    return STEPQ_OK;
}

stepq_status stepq_setup_distortion(int64_t C, int32_t H, int32_t d_k, int32_t d_v, const float *states,
                                    const float *row_weight, const uint8_t *pivots, int32_t n_cand,
                                    const int32_t *cand_bits, int32_t unit, double *d_out, int32_t n_threads)
{
    if (C < 1 || H < 1 || d_k < 1 || d_v < 1 || !states || n_cand < 1 || !cand_bits || !d_out) return STEPQ_E_INVALID;
    if (unit != 0 && unit != 1) return STEPQ_E_INVALID;
    for (int32_t ci = 0; ci < n_cand; ++ci)
        if (cand_bits[ci] != 2 && cand_bits[ci] != 4 && cand_bits[ci] != 8 && cand_bits[ci] != 16)
            return STEPQ_E_INVALID;
    const size_t nel = static_cast<size_t>(d_k) * d_v;
    // squared error per (candidate, head, row), summed over samples and columns
    std::vector<double> err(static_cast<size_t>(n_cand) * H * d_k, 0.0);
    std::mutex mu;
    parallel_for(C * H, n_threads, [&](int64_t a, int64_t b) {
        std::vector<double> loc(err.size(), 0.0), X(nel), R(nel), w(d_k), r, c;
        std::vector<uint8_t> bits(d_k);
        for (int64_t sh = a; sh < b; ++sh) {
            const int32_t h = static_cast<int32_t>(sh % H);
            const float *S = states + static_cast<size_t>(sh) * nel;
            for (size_t e = 0; e < nel; ++e) X[e] = static_cast<double>(S[e]);
            for (int32_t i = 0; i < d_k; ++i)
                w[i] = row_weight ? static_cast<double>(row_weight[static_cast<size_t>(h) * d_k + i]) : 1.0;
            for (int32_t ci = 0; ci < n_cand; ++ci) {
                const int32_t bc = cand_bits[ci];
                for (int32_t i = 0; i < d_k; ++i)
                    bits[i] = (bc == 16 || (pivots && pivots[static_cast<size_t>(h) * d_k + i])) ? 16 : bc;
                codec_tile(d_k, d_v, X.data(), bits.data(), w.data(), R.data(), r, c);
                for (int32_t i = 0; i < d_k; ++i) {
                    double s = 0.0;
                    for (int32_t j = 0; j < d_v; ++j) {
                        const double dd = R[static_cast<size_t>(i) * d_v + j] - X[static_cast<size_t>(i) * d_v + j];
                        s += dd * dd;
                    }
                    loc[(static_cast<size_t>(ci) * H + h) * d_k + i] += s;
                }
            }
        }
        std::lock_guard<std::mutex> lk(mu);
        for (size_t e = 0; e < err.size(); ++e) err[e] += loc[e];
    });
    for (int32_t h = 0; h < H; ++h) {
        if (unit == 0) {           // key rows: unweighted MSE per row
            for (int32_t i = 0; i < d_k; ++i)
                for (int32_t ci = 0; ci < n_cand; ++ci)
                    d_out[(static_cast<size_t>(h) * d_k + i) * n_cand + ci] =
                        err[(static_cast<size_t>(ci) * H + h) * d_k + i] / (static_cast<double>(C) * d_v);
        } else {                   // heads: w^2-weighted MSE over the head
            for (int32_t ci = 0; ci < n_cand; ++ci) {
                double s = 0.0;
                for (int32_t i = 0; i < d_k; ++i) {
                    const double wi = row_weight ? static_cast<double>(row_weight[static_cast<size_t>(h) * d_k + i]) : 1.0;
                    s += wi * wi * err[(static_cast<size_t>(ci) * H + h) * d_k + i];
                }
                d_out[static_cast<size_t>(h) * n_cand + ci] = s / (static_cast<double>(C) * d_k * d_v);
            }
        }
    }
    return STEPQ_OK;
}

stepq_status stepq_setup_lifetime_weights(int32_t U, const double *ell, int32_t horizon, double *L)
{
    if (U < 1 || !ell || !L || horizon < 1) return STEPQ_E_INVALID;
    for (int32_t u = 0; u < U; ++u) {
        // sum_{j<H} exp(2 j l) as the geometric series it is (terms summed when l = 0)
        const double x = 2.0 * ell[u];
        L[u] = std::fabs(x) < 1e-12 ? static_cast<double>(horizon)
                                     : std::expm1(x * horizon) / std::expm1(x);
    }
    return STEPQ_OK;
}

stepq_status stepq_setup_mean_log_retention(int64_t T, int32_t H, int32_t d_k, const float *gate, int32_t gate_per_row,
                                            int32_t unit, double *ell)
{
    if (T < 1 || H < 1 || d_k < 1 || !gate || !ell || (gate_per_row != 0 && gate_per_row != 1) ||
        (unit != 0 && unit != 1))
        return STEPQ_E_INVALID;
    const int64_t per_t = gate_per_row ? static_cast<int64_t>(H) * d_k : H;
    for (int64_t e = 0; e < T * per_t; ++e)
        if (!(gate[e] > 0.0f) || !std::isfinite(gate[e])) return STEPQ_E_INVALID;
    // per key row: the mean over samples of log of the row's gate (its own
    // channel under a channel-wise gate, its head's otherwise)
    std::vector<double> rows(static_cast<size_t>(H) * d_k, 0.0);
    for (int32_t h = 0; h < H; ++h)
        for (int32_t i = 0; i < d_k; ++i) {
            double s = 0.0;
            for (int64_t t = 0; t < T; ++t)
                s += std::log(static_cast<double>(gate_per_row ? gate[(t * H + h) * d_k + i] : gate[t * H + h]));
            rows[static_cast<size_t>(h) * d_k + i] = s / static_cast<double>(T);
        }
    if (unit == 0) {
        std::copy(rows.begin(), rows.end(), ell);
    } else {
        // a head unit: the mean over its rows
        for (int32_t h = 0; h < H; ++h) {
            double s = 0.0;
            for (int32_t i = 0; i < d_k; ++i) s += rows[static_cast<size_t>(h) * d_k + i];
            ell[h] = s / static_cast<double>(d_k);
        }
    }
    return STEPQ_OK;
}

stepq_status stepq_setup_lifetime_costs(int32_t U, int32_t n_cand, const double *L, const double *d, int32_t d_stride,
                                        double *cost)
{
    if (U < 1 || n_cand < 1 || d_stride < n_cand || !L || !d || !cost) return STEPQ_E_INVALID;
    for (int32_t u = 0; u < U; ++u)
        for (int32_t c = 0; c < n_cand; ++c)
            cost[static_cast<size_t>(u) * n_cand + c] = L[u] * d[static_cast<size_t>(u) * d_stride + c];
    return STEPQ_OK;
}

stepq_status stepq_setup_pivot_risk(int32_t U, const double *L, const double *d, int32_t d_stride, int32_t col_int,
                                    int32_t col_f16, double *risk)
{
    if (U < 1 || !L || !d || !risk || col_int < 0 || col_f16 < 0 || col_int >= d_stride || col_f16 >= d_stride)
        return STEPQ_E_INVALID;
    for (int32_t u = 0; u < U; ++u)
        risk[u] = L[u] * (d[static_cast<size_t>(u) * d_stride + col_int] - d[static_cast<size_t>(u) * d_stride + col_f16]);
    return STEPQ_OK;
}

stepq_status stepq_setup_select_pivots(int32_t U, const double *risk, int32_t count, uint8_t *is_pivot)
{
    if (U < 1 || !risk || !is_pivot || count < 0 || count > U) return STEPQ_E_INVALID;
    std::vector<int32_t> order(U);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return risk[a] > risk[b]; });
    std::fill(is_pivot, is_pivot + U, 0);
    for (int32_t k = 0; k < count; ++k) is_pivot[order[k]] = 1;
    return STEPQ_OK;
}

stepq_status stepq_setup_allocate(int32_t U, int32_t n_cand, const int32_t *cand_bits, const double *cost,
                                  const int32_t *n_u, double budget, int32_t method, int32_t *choice)
{
    if (U < 1 || n_cand < 1 || !cand_bits || !cost || !n_u || !choice || (method != 0 && method != 1))
        return STEPQ_E_INVALID;
    double total = 0.0;
    for (int32_t u = 0; u < U; ++u) {
        if (n_u[u] < 1) return STEPQ_E_INVALID;
        total += n_u[u];
    }
    for (int32_t ci = 0; ci < n_cand; ++ci)
        if (cand_bits[ci] < 1) return STEPQ_E_INVALID;
    const double cap = budget * total;
    auto c_at = [&](int32_t u, int32_t ci) { return cost[static_cast<size_t>(u) * n_cand + ci]; };
    if (method == 0) {
        // multiple-choice knapsack: exact DP over spent bits in gcd units
        int64_t g = 0;
        for (int32_t u = 0; u < U; ++u)
            for (int32_t ci = 0; ci < n_cand; ++ci) g = std::gcd(g, static_cast<int64_t>(n_u[u]) * cand_bits[ci]);
        const int64_t capu = static_cast<int64_t>(std::floor(cap / static_cast<double>(g) + 1e-9));
        if (capu < 0) return STEPQ_E_INVALID;
        if (static_cast<double>(capu + 1) * U > 4e8) return STEPQ_E_UNSUPPORTED;     // use the Lagrangian
        const double INF = std::numeric_limits<double>::infinity();
        std::vector<double> best(capu + 1, INF), nxt(capu + 1);
        std::vector<int8_t> pick(static_cast<size_t>(U) * (capu + 1), -1);
        best[0] = 0.0;
        for (int32_t u = 0; u < U; ++u) {
            std::fill(nxt.begin(), nxt.end(), INF);
            int8_t *pk = pick.data() + static_cast<size_t>(u) * (capu + 1);
            for (int64_t s = 0; s <= capu; ++s) {
                if (best[s] == INF) continue;
                for (int32_t ci = 0; ci < n_cand; ++ci) {
                    const int64_t s2 = s + static_cast<int64_t>(n_u[u]) * cand_bits[ci] / g;
                    const double v = best[s] + c_at(u, ci);
                    if (s2 <= capu && v < nxt[s2]) {
                        nxt[s2] = v;
                        pk[s2] = static_cast<int8_t>(ci);
                    }
                }
            }
            best.swap(nxt);
        }
        int64_t se = -1;
        for (int64_t s = 0; s <= capu; ++s)
            if (best[s] < INF && (se < 0 || best[s] < best[se])) se = s;
        if (se < 0) return STEPQ_E_INVALID;           // no assignment fits the budget
        for (int32_t u = U - 1; u >= 0; --u) {
            const int32_t ci = pick[static_cast<size_t>(u) * (capu + 1) + se];
            choice[u] = ci;
            se -= static_cast<int64_t>(n_u[u]) * cand_bits[ci] / g;
        }
        return STEPQ_OK;
    }
    // Lagrangian: per unit argmin cost + lam n_u b (ties: the narrower), the
    // smallest lam that fits by bisection, then greedy repair
    auto assign = [&](double lam, std::vector<int32_t> &ch) {
        double spent = 0.0;
        for (int32_t u = 0; u < U; ++u) {
            int32_t bi = 0;
            double bv = c_at(u, 0) + lam * n_u[u] * cand_bits[0];
            for (int32_t ci = 1; ci < n_cand; ++ci) {
                const double v = c_at(u, ci) + lam * n_u[u] * cand_bits[ci];
                if (v < bv || (v == bv && cand_bits[ci] < cand_bits[bi])) {
                    bv = v;
                    bi = ci;
                }
            }
            ch[u] = bi;
            spent += static_cast<double>(n_u[u]) * cand_bits[bi];
        }
        return spent;
    };
    std::vector<int32_t> ch(U);
    double lo = 0.0, hi = 1.0;
    while (assign(hi, ch) > cap) {
        hi *= 2.0;
        if (hi > 1e300) return STEPQ_E_INVALID;        // below the narrowest assignment
    }
    if (assign(lo, ch) > cap) {
        for (int it = 0; it < 200; ++it) {
            const double mid = 0.5 * (lo + hi);
            if (assign(mid, ch) <= cap) hi = mid;
            else lo = mid;
        }
        assign(hi, ch);
    }
    for (;;) {
        double spent = 0.0;
        for (int32_t u = 0; u < U; ++u) spent += static_cast<double>(n_u[u]) * cand_bits[ch[u]];
        const double left = cap - spent;
        double bestg = 0.0;
        int32_t bu = -1, bc = -1;
        for (int32_t u = 0; u < U; ++u)
            for (int32_t ci = 0; ci < n_cand; ++ci) {
                const double extra = static_cast<double>(n_u[u]) * (cand_bits[ci] - cand_bits[ch[u]]);
                if (extra <= 0.0 || extra > left + 1e-9) continue;
                const double gain = (c_at(u, ch[u]) - c_at(u, ci)) / extra;
                if (gain > bestg) {
                    bestg = gain;
                    bu = u;
                    bc = ci;
                }
            }
        if (bu < 0) break;
        ch[bu] = bc;
    }
    std::copy(ch.begin(), ch.end(), choice);
    return STEPQ_OK;
}

}  // extern "C"
