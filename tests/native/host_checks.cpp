// Host code of libstepq under the CPU sanitizers (AddressSanitizer and
// UndefinedBehaviorSanitizer, built by tests/test_sanitizers.py): the layout
// derivation and launch planning of stepq_plan.cpp, including plans
// corrupted on purpose, which the plan check must refuse; the multiply-high
// division constants the kernels use; and every call of the CPU setup step
// on small random inputs and on its error paths.  Exits non-zero on the
// first failed expectation.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "stepq.h"
#include "stepq_plan.h"

namespace {

int g_failures = 0;

void expect(bool ok, const char *what, const std::string &detail = "")
{
    if (!ok) {
        std::fprintf(stderr, "FAILED: %s %s\n", what, detail.c_str());
        ++g_failures;
    }
}

struct Rng {
    uint64_t s;
    explicit Rng(uint64_t seed) : s(seed * 0x9E3779B97F4A7C15ull + 1) {}
    uint64_t next()
    {
        s ^= s << 13;
        s ^= s >> 7;
        s ^= s << 17;
        return s;
    }
    int below(int n) { return static_cast<int>(next() % static_cast<uint64_t>(n)); }
    double unit() { return (next() >> 11) * (1.0 / 9007199254740992.0); }
    double normal()
    {
        const double u = unit() + 1e-300, v = unit();
        return std::sqrt(-2.0 * std::log(u)) * std::cos(6.283185307179586 * v);
    }
};

// One head's row widths by recipe: uniform mixes (shuffled), a mix with a
// few pivot rows, a whole FP16 head, an irregular 8/4 split, random widths.
void head_bits(Rng &g, int recipe, int dk, uint8_t *b)
{
    static const int mixes[5][3] = {{64, 64, 0}, {32, 32, 64}, {128, 0, 0}, {0, 128, 0}, {0, 0, 128}};
    for (int i = 0; i < dk; ++i) b[i] = static_cast<uint8_t>(2 << g.below(3));
    if (dk != 128) return;
    if (recipe <= 1) {
        const int *m = mixes[g.below(5)];
        int i = 0;
        for (int w = 0; w < 3; ++w)
            for (int c = 0; c < m[w]; ++c) b[i++] = static_cast<uint8_t>(8 >> w);
        if (recipe == 1)
            for (int p = 1 + g.below(8); p > 0; --p) b[g.below(dk)] = 16;
    } else if (recipe == 2) {
        for (int i = 0; i < dk; ++i) b[i] = 16;
    } else if (recipe == 3) {
        const int n8 = 40 + g.below(50);
        for (int i = 0; i < dk; ++i) b[i] = i < n8 ? 8 : 4;
        for (int p = g.below(6); p > 0; --p) b[g.below(dk)] = 16;
    }
    for (int i = dk - 1; i > 0; --i) std::swap(b[i], b[g.below(i + 1)]);
}

void check_plans()
{
    Rng g(1);
    int mixed = 0, combined = 0, single = 0;
    for (int trial = 0; trial < 3000; ++trial) {
        const int dv = g.below(4) == 0 ? 64 : 128;
        const int dk = g.below(3) == 0 ? 1 + g.below(128) : 128;
        const int Hv = 1 + g.below(40);
        std::vector<uint8_t> bits(static_cast<size_t>(Hv) * dk);
        const int recipes = 1 + g.below(3);
        int pool_recipe[3];
        for (int r = 0; r < recipes; ++r) pool_recipe[r] = g.below(5);
        for (int h = 0; h < Hv; ++h) head_bits(g, pool_recipe[g.below(recipes)], dk, &bits[static_cast<size_t>(h) * dk]);
        stepq_pool_desc d{1 + g.below(9), Hv, 1, dk, dv, bits.data(), g.below(2)};
        std::vector<stepq::HeadInfo> heads;
        std::vector<uint8_t> perm;
        size_t sb = 0;
        std::string err;
        if (stepq::derive_layout(&d, &heads, &perm, &sb, &err) != STEPQ_OK) {
            // only over-long pivot lists are refused
            expect(err.find("pivot") != std::string::npos, "derive_layout refused a valid map", err);
            continue;
        }
        stepq::LaunchPlan plan;
        stepq::plan_launches(heads, dk, dv, &plan);
        expect(stepq::check_plan(plan, heads, dk, dv, sb, &err), "plan of a valid descriptor refused", err);
        if (plan.order.empty()) {
            ++single;
            stepq::LaunchPlan bad = plan;
            bad.layout = plan.layout == 1 ? 2 : 1;
            expect(!stepq::check_plan(bad, heads, dk, dv, sb, &err), "single launch with another layout accepted");
            continue;
        }
        ++mixed;
        combined += plan.mixed_code != 0;
        // corrupted plans must all be refused
        auto refused = [&](const stepq::LaunchPlan &p, const char *what) {
            expect(!stepq::check_plan(p, heads, dk, dv, sb, &err), what);
        };
        const int e = g.below(Hv);
        stepq::LaunchPlan bad = plan;
        bad.order[e].h = Hv;
        refused(bad, "head index out of range accepted");
        if (Hv > 1) {
            bad = plan;
            bad.order[e].h = plan.order[(e + 1) % Hv].h;
            refused(bad, "a head listed twice accepted");
        }
        bad = plan;
        bad.order[e].tile_off += 128;
        refused(bad, "a wrong tile offset accepted");
        bad = plan;
        bad.order[e].counts ^= 1 << 8;
        refused(bad, "wrong row counts accepted");
        bad = plan;
        bad.cls_cnt.back() += 1;
        refused(bad, "a class running past the head list accepted");
        if (plan.cls_cnt.size() > 1) {
            bad = plan;
            bad.cls_cnt[1] = Hv;    // a class launch given the whole pool's head count
            refused(bad, "a class launch over more heads than its class accepted");
        }
        bad = plan;
        bad.cls_code[0] = plan.cls_code[0] == 1 ? 2 : 1;
        refused(bad, "a class given a body that does not run its heads accepted");
        bool non_compiled = false;
        for (int c : plan.cls_code) non_compiled = non_compiled || !(c >= 1 && c <= stepq::kF16HeadLayout);
        if (non_compiled) {
            bad = plan;
            bad.mixed_code = stepq::kMultiUniform;
            refused(bad, "a combined launch over heads its body does not run accepted");
        }
        std::vector<stepq::HeadInfo> grown = heads;
        grown.back().tile_bytes += 128;
        expect(!stepq::check_plan(plan, grown, dk, dv, sb, &err), "a tile past the slot record accepted");
    }
    expect(single > 100 && mixed > 100 && combined > 20, "plan cases not all reached",
           std::to_string(single) + " " + std::to_string(mixed) + " " + std::to_string(combined));
    std::printf("plans: %d single-launch, %d with head lists (%d combined)\n", single, mixed, combined);
}

void check_fast_div()
{
    Rng g(2);
    for (uint32_t d = 1; d <= 4096; ++d) {
        const stepq::FastDiv f = stepq::fast_div(d);
        auto q = [&](uint32_t n) {
            return static_cast<uint32_t>((((static_cast<uint64_t>(n) * f.mul) >> 32) + n) >> f.shift);
        };
        for (uint32_t n = 0; n < 4096; ++n) expect(q(n) == n / d, "fast_div small numerator");
        for (uint64_t k = 1; k * d < (1ull << 31); k = k * 3 + 1) {
            const uint32_t n = static_cast<uint32_t>(k * d);
            expect(q(n) == k && q(n - 1) == (n - 1) / d, "fast_div at a multiple");
        }
        for (int t = 0; t < 64; ++t) {
            const uint32_t n = static_cast<uint32_t>(g.next() & 0x7fffffffu);
            expect(q(n) == n / d, "fast_div random numerator");
        }
        expect(q(0x7fffffffu) == 0x7fffffffu / d, "fast_div largest numerator");
    }
}

void check_setup()
{
    Rng g(3);
    const int n = 3, dk = 17, dv = 64;
    std::vector<float> S(static_cast<size_t>(n) * dk * dv), w(n * dk), r(n * dk), c(n * dv);
    for (auto &x : S) x = static_cast<float>(g.normal() * std::exp(g.normal()));
    for (int j = 0; j < dv; ++j) S[5 * dv + j] = 0.0f;       // an all-zero row
    for (auto &x : w) x = static_cast<float>(std::exp(0.5 * g.normal()));
    std::vector<uint8_t> bits(n * dk);
    for (auto &b : bits) b = static_cast<uint8_t>(g.below(6) == 0 ? 16 : 2 << g.below(3));
    for (int levels = 0; levels < 2; ++levels) {
        expect(stepq_setup_fit_levels(n, dk, dv, S.data(), w.data(), bits.data(), levels, r.data(), c.data(), 2) ==
                   STEPQ_OK, "stepq_setup_fit_levels");
        for (int t = 0; t < n; ++t)
            for (int i = 0; i < dk; ++i) {
                const int b = bits[t * dk + i];
                if (b == 16) continue;
                const double qb = (1 << (b - 1)) - 1;
                const double top = levels ? qb * std::ldexp(1.0, 8 - b) : 1.0;
                for (int j = 0; j < dv; ++j)
                    expect(static_cast<double>(r[t * dk + i]) * c[t * dv + j] * top >=
                               std::fabs(S[(static_cast<size_t>(t) * dk + i) * dv + j]),
                           "fitted scales bound the state");
            }
    }
    expect(stepq_setup_fit(n, dk, dv, S.data(), nullptr, r.data(), c.data(), 0) == STEPQ_OK, "stepq_setup_fit");
    expect(stepq_setup_fit(n, dk, dv, nullptr, nullptr, r.data(), c.data(), 0) == STEPQ_E_INVALID,
           "stepq_setup_fit refuses NULL");
    expect(stepq_setup_fit_levels(n, dk, dv, S.data(), nullptr, nullptr, 1, r.data(), c.data(), 1) ==
               STEPQ_E_INVALID, "N2 fit needs row widths");

    const int T = 5, B = 3, H = 4;
    std::vector<double> gates(T * B * H);
    for (auto &x : gates) x = 0.8 + 0.19 * g.unit();
    std::vector<uint8_t> rb(H * dk);
    expect(stepq_setup_lifetime_bits(gates.data(), T, B, H, dk, 6.0, 4, 8, rb.data()) == STEPQ_OK,
           "stepq_setup_lifetime_bits");
    int wide = 0;
    for (uint8_t b : rb) wide += b == 8;
    expect(wide == H * dk / 2, "lifetime bits meet the budget");

    const int Tc = 7;
    std::vector<float> q(Tc * H * dk), k(Tc * H * dk), beta(Tc * H), gate(Tc * H * dk), rw(H * dk);
    for (auto &x : q) x = static_cast<float>(g.normal());
    for (auto &x : k) x = static_cast<float>(g.normal());
    for (auto &x : beta) x = static_cast<float>(g.unit());
    for (auto &x : gate) x = static_cast<float>(0.5 + 0.5 * g.unit());
    std::vector<double> omega(H * dk);
    for (int per_row = 0; per_row < 2; ++per_row)
        expect(stepq_setup_row_impact(Tc, H, dk, q.data(), k.data(), beta.data(), gate.data(), per_row, 0.25,
                                      rw.data(), omega.data()) == STEPQ_OK, "stepq_setup_row_impact");
    for (float x : rw) expect(std::isfinite(x) && x > 0.0f, "row weights finite and positive");

    const int C = 2;
    std::vector<float> states(static_cast<size_t>(C) * H * dk * dv);
    for (auto &x : states) x = static_cast<float>(0.05 * g.normal());
    std::vector<uint8_t> piv(H * dk, 0);
    piv[3] = piv[dk + 7] = 1;
    const int cand[4] = {2, 4, 8, 16};
    std::vector<double> dist_rows(H * dk * 4), dist_heads(H * 4);
    expect(stepq_setup_distortion(C, H, dk, dv, states.data(), rw.data(), piv.data(), 4, cand, 0, dist_rows.data(),
                                  2) == STEPQ_OK, "stepq_setup_distortion rows");
    expect(stepq_setup_distortion(C, H, dk, dv, states.data(), nullptr, nullptr, 4, cand, 1, dist_heads.data(), 0) ==
               STEPQ_OK, "stepq_setup_distortion heads");
    const int bad6[1] = {6};
    expect(stepq_setup_distortion(C, H, dk, dv, states.data(), nullptr, nullptr, 1, bad6, 1, dist_heads.data(), 0) ==
               STEPQ_E_INVALID, "a 6-bit candidate is refused");
    for (double x : dist_rows) expect(std::isfinite(x) && x >= 0.0, "row distortions finite");

    const int U = H * dk;
    std::vector<double> ell(U), L(U);
    for (auto &x : ell) x = std::log(0.8 + 0.19 * g.unit());
    expect(stepq_setup_lifetime_weights(U, ell.data(), 64, L.data()) == STEPQ_OK, "stepq_setup_lifetime_weights");
    std::vector<double> cost(U * 3);
    for (int u = 0; u < U; ++u)
        for (int x = 0; x < 3; ++x) cost[u * 3 + x] = L[u] * dist_rows[u * 4 + x];
    std::vector<int32_t> nu(U, dv), choice(U);
    for (int method = 0; method < 2; ++method) {
        expect(stepq_setup_allocate(U, 3, cand, cost.data(), nu.data(), 4.0, method, choice.data()) == STEPQ_OK,
               "stepq_setup_allocate");
        double spent = 0;
        for (int u = 0; u < U; ++u) spent += cand[choice[u]];
        expect(spent <= 4.0 * U + 1e-9, "allocation within budget");
    }
    expect(stepq_setup_allocate(U, 3, cand, cost.data(), nu.data(), 1.0, 0, choice.data()) == STEPQ_E_INVALID,
           "an unreachable budget is refused");
    std::vector<uint8_t> is_piv(U);
    expect(stepq_setup_select_pivots(U, L.data(), 5, is_piv.data()) == STEPQ_OK, "stepq_setup_select_pivots");
    int np = 0;
    for (uint8_t x : is_piv) np += x;
    expect(np == 5, "pivot count");
}

}  // namespace

int main()
{
    check_plans();
    check_fast_div();
    check_setup();
    if (g_failures) {
        std::fprintf(stderr, "%d failed expectations\n", g_failures);
        return 1;
    }
    std::printf("host checks ok\n");
    return 0;
}
