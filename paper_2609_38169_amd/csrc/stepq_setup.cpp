// CPU setup step of libstepq (offline, host memory only): the dual-axis
// scale fit of the initial states and the lifetime-ranked bit allocation.
#include <algorithm>
#include <cmath>
#include <numeric>
#include <string>
#include <thread>
#include <vector>

#include "stepq.h"

namespace {

void fit_tiles(int64_t t0, int64_t t1, int32_t dk, int32_t dv, const float *S, const float *w, const uint8_t *bits,
               float *r, float *c)
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
            for (int j = 0; j < dv; ++j) {
                const double a = std::fabs(static_cast<double>(row[j])) / inv;
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
    if (n_tiles < 0 || d_k < 1 || d_v < 1) return STEPQ_E_INVALID;
    if (n_tiles == 0) return STEPQ_OK;
    if (!state || !r || !c) return STEPQ_E_INVALID;
    int nt = n_threads > 0 ? n_threads : static_cast<int>(std::max(1u, std::thread::hardware_concurrency()));
    nt = static_cast<int>(std::min<int64_t>(nt, n_tiles));
    if (nt <= 1) {
        fit_tiles(0, n_tiles, d_k, d_v, state, row_weight, row_bits, r, c);
        return STEPQ_OK;
    }
    std::vector<std::thread> pool;
    const int64_t per = (n_tiles + nt - 1) / nt;
    for (int k = 0; k < nt; ++k) {
        const int64_t t0 = k * per, t1 = std::min<int64_t>(n_tiles, t0 + per);
        if (t0 >= t1) break;
        pool.emplace_back(fit_tiles, t0, t1, d_k, d_v, state, row_weight, row_bits, r, c);
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

}  // extern "C"
