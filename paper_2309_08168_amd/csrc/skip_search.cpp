// Skip-set search (Sec. 3.3, Eq. 1): z* = argmin f(z) over the masks z in
// {0, 1}^L of sublayers the draft bypasses, f the time per emitted token.
// Bayesian optimisation as the paper describes it: a Gaussian-process
// surrogate of f and an acquisition (expected improvement) choose the next
// mask to evaluate, for a fixed number of steps.
//
// The surrogate's factor grows by one row per evaluation: the kernel matrix
// of the observed masks never changes, only the standardised observations
// do, so each step costs O(n^2) per candidate plus O(n^2) for the new
// weights, and the factor is never rebuilt.  Masks are packed 64 to a word
// for the Hamming distances; kernel values come from a table over the
// distance.
//
// Host code only: the objective of sd_search_skip_set runs the library's
// self-speculative decoding on the GPU.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <new>
#include <string>
#include <unordered_set>
#include <vector>

#include "host_api.h"
#include "sd.h"

namespace {

using sdk::report;

constexpr int32_t MAX_DIMS = 1024;
constexpr int32_t MAX_EVALS = 4096;
constexpr int32_t MAX_CANDIDATES = 65536;

// Purposes of the search's uniforms (second counter word).
enum : uint64_t { P_INIT = 100, P_NFLIP = 101, P_FLIP = 102, P_DENSITY = 103, P_BIT = 104 };

// Philox4x64-10 (Salmon et al., SC'11, the 4x64 variant's multipliers and
// Weyl constants) under key (seed, 1); the top 24 bits of the first output
// word as a uniform on [0, 1).
double search_uniform(uint64_t seed, uint64_t a, uint64_t purpose, uint64_t c) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
    uint64_t x0 = a, x1 = purpose, x2 = c, x3 = 0, k0 = seed, k1 = 1;
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += W0;
            k1 += W1;
        }
        const unsigned __int128 p0 = (unsigned __int128)M0 * x0, p1 = (unsigned __int128)M1 * x2;
        const uint64_t n0 = (uint64_t)(p1 >> 64) ^ x1 ^ k0, n2 = (uint64_t)(p0 >> 64) ^ x3 ^ k1;
        x1 = (uint64_t)p1;
        x3 = (uint64_t)p0;
        x0 = n0;
        x2 = n2;
    }
    return (double)(x0 >> 40) * 0x1p-24;
}

// A mask as bytes (the ABI's layout) and as packed bits.
struct Mask {
    std::vector<uint8_t> bytes;
    std::vector<uint64_t> bits;

    explicit Mask(int32_t L) : bytes(L, 0), bits((L + 63) / 64, 0) {}
    void set(int32_t j, bool v) {
        bytes[j] = v;
        const uint64_t b = 1ull << (j % 64);
        bits[j / 64] = v ? (bits[j / 64] | b) : (bits[j / 64] & ~b);
    }
    bool operator==(const Mask &o) const { return bits == o.bits; }
};

struct MaskHash {
    size_t operator()(const Mask &m) const {
        uint64_t h = 0x9E3779B97F4A7C15ull;
        for (uint64_t w : m.bits)
            h = (h ^ w) * 0xBF58476D1CE4E5B9ull;
        return (size_t)(h ^ (h >> 31));
    }
};

int hamming(const Mask &a, const Mask &b) {
    int h = 0;
    for (size_t i = 0; i < a.bits.size(); ++i)
        h += __builtin_popcountll(a.bits[i] ^ b.bits[i]);
    return h;
}

Mask initial_mask(uint64_t seed, int32_t i, int32_t n_init, int32_t L) {
    Mask z(L);
    const double p = 0.6 * i / n_init;  // mask 0 is empty: the full model as its own draft
    for (int32_t j = 0; j < L; ++j)
        z.set(j, search_uniform(seed, i, P_INIT, j) < p);
    return z;
}

// Candidate c of step t: the first half flip 1 to 3 bits of the incumbent,
// the rest are random masks of one random density in [0, 0.6).
Mask candidate(uint64_t seed, int32_t t, int32_t c, int32_t n_cand, int32_t L, const Mask &incumbent) {
    if (c < n_cand / 2) {
        Mask z = incumbent;
        const int flips = 1 + (int)(search_uniform(seed, t, P_NFLIP, c) * 3.0);
        for (int r = 0; r < flips; ++r) {
            const int32_t j = (int32_t)(search_uniform(seed, t, P_FLIP, (uint64_t)c * 8 + r) * L);
            z.set(j, !z.bytes[j]);
        }
        return z;
    }
    Mask z(L);
    const double p = 0.6 * search_uniform(seed, t, P_DENSITY, c);
    for (int32_t j = 0; j < L; ++j)
        z.set(j, search_uniform(seed, t, P_BIT, (uint64_t)c * L + j) < p);
    return z;
}

// Gaussian process over the observed masks: the lower Cholesky factor of
// K + noise I (packed rows), extended by one row per observation.
class Surrogate {
  public:
    Surrogate(int32_t L, double length_scale, double noise, int32_t cap) : noise_(noise) {
        ktab_.resize(L + 1);
        for (int32_t h = 0; h <= L; ++h)
            ktab_[h] = std::exp(-(double)h / (length_scale * L));
        fac_.reserve((size_t)cap * (cap + 1) / 2);
        X_.reserve(cap);
    }

    int32_t size() const { return (int32_t)X_.size(); }
    const Mask &mask(int32_t i) const { return X_[i]; }

    // Appends mask z; false when the extended matrix is not positive definite.
    bool add(const Mask &z) {
        const int32_t n = size();
        std::vector<double> v(n);
        kvec(z, v.data());
        solve_lower(v.data());
        double d = 1.0 + noise_;
        for (int32_t i = 0; i < n; ++i)
            d -= v[i] * v[i];
        if (!(d > 0.0))
            return false;
        fac_.insert(fac_.end(), v.begin(), v.end());
        fac_.push_back(std::sqrt(d));
        X_.push_back(z);
        return true;
    }

    // Weights alpha = (K + noise I)^-1 ys of the standardised observations.
    void set_observations(const std::vector<double> &ys) {
        alpha_ = ys;
        solve_lower(alpha_.data());
        solve_upper(alpha_.data());
    }

    // Posterior mean and standard deviation of the noise-free value at z;
    // work holds size() doubles.
    void predict(const Mask &z, double *work, double *mu, double *sigma) const {
        const int32_t n = size();
        kvec(z, work);
        double m = 0.0;
        for (int32_t i = 0; i < n; ++i)
            m += work[i] * alpha_[i];
        solve_lower(work);
        double v = 1.0;
        for (int32_t i = 0; i < n; ++i)
            v -= work[i] * work[i];
        *mu = m;
        *sigma = std::sqrt(std::max(v, 0.0));
    }

  private:
    const double *row(int32_t i) const { return fac_.data() + (size_t)i * (i + 1) / 2; }

    void kvec(const Mask &z, double *k) const {
        for (int32_t i = 0; i < size(); ++i)
            k[i] = ktab_[hamming(z, X_[i])];
    }
    void solve_lower(double *b) const {  // b <- F^-1 b
        for (int32_t i = 0; i < size(); ++i) {
            const double *r = row(i);
            double s = b[i];
            for (int32_t k = 0; k < i; ++k)
                s -= r[k] * b[k];
            b[i] = s / r[i];
        }
    }
    void solve_upper(double *b) const {  // b <- F^-T b
        for (int32_t i = size() - 1; i >= 0; --i) {
            const double *r = row(i);
            b[i] /= r[i];
            for (int32_t k = 0; k < i; ++k)
                b[k] -= r[k] * b[i];
        }
    }

    double noise_;
    std::vector<double> ktab_, fac_, alpha_;
    std::vector<Mask> X_;
};

std::vector<double> standardise(const std::vector<double> &y) {
    const size_t n = y.size();
    double mean = 0.0;
    for (double v : y)
        mean += v;
    mean /= (double)n;
    double ss = 0.0;
    for (double v : y)
        ss += (v - mean) * (v - mean);
    double sd = std::sqrt(ss / (double)n);
    if (!(sd > 1e-12))
        sd = 1.0;
    std::vector<double> ys(n);
    for (size_t i = 0; i < n; ++i)
        ys[i] = (y[i] - mean) / sd;
    return ys;
}

// Expected improvement (minimisation) below best by xi.
double expected_improvement(double mu, double sigma, double best, double xi) {
    const double imp = best - mu - xi;
    if (!(sigma > 0.0))
        return std::max(imp, 0.0);
    const double u = imp / sigma;
    const double cdf = 0.5 * std::erfc(-u / std::sqrt(2.0));
    const double pdf = std::exp(-0.5 * u * u) / std::sqrt(2.0 * M_PI);
    return imp * cdf + sigma * pdf;
}

sd_status check_params(int32_t L, const sd_search_params *p, const sd_search_result *res) {
    if (!p || !res || !res->best_mask)
        return report(SD_ERR_INVALID_ARG, "params, result and result->best_mask are required");
    if (L < 1 || L > MAX_DIMS)
        return report(SD_ERR_INVALID_ARG, "the mask must have 1 to 1024 entries");
    if (p->n_init < 1 || p->iterations < 0 || (int64_t)p->n_init + p->iterations > MAX_EVALS)
        return report(SD_ERR_INVALID_ARG, "need n_init >= 1, iterations >= 0, n_init + iterations <= 4096");
    if (p->n_candidates < 1 || p->n_candidates > MAX_CANDIDATES)
        return report(SD_ERR_INVALID_ARG, "n_candidates must be in [1, 65536]");
    if (!(p->length_scale > 0.0) || !std::isfinite(p->length_scale) || !(p->noise > 0.0) ||
        !std::isfinite(p->noise) || !std::isfinite(p->xi))
        return report(SD_ERR_INVALID_ARG, "need finite length_scale > 0, noise > 0 and xi");
    return SD_OK;
}

using Objective = sd_status (*)(const uint8_t *, int32_t, void *, double *);

sd_status run_search(int32_t L, const sd_search_params &p, Objective objective, void *user,
                     sd_search_result *res) {
    const int32_t cap = p.n_init + p.iterations;
    Surrogate gp(L, p.length_scale, p.noise, cap);
    std::unordered_set<Mask, MaskHash> seen;
    std::vector<double> y;
    y.reserve(cap);
    int32_t evals = 0;

    auto evaluate = [&](const Mask &z, double margin) -> sd_status {
        double v = 0.0;
        const sd_status rc = objective(z.bytes.data(), L, user, &v);
        if (rc != SD_OK)
            return report(rc, "objective failed at evaluation " + std::to_string(evals) + ": " + sd_last_error());
        if (!std::isfinite(v))
            return report(SD_ERR_INVALID_ARG, "objective returned a non-finite value");
        if (!gp.add(z))
            return report(SD_ERR_INVALID_ARG, "surrogate matrix is not positive definite (raise noise)");
        seen.insert(z);
        y.push_back(v);
        if (res->masks)
            std::memcpy(res->masks + (size_t)evals * L, z.bytes.data(), L);
        if (res->values)
            res->values[evals] = v;
        if (res->margins)
            res->margins[evals] = margin;
        ++evals;
        res->n_evaluated = evals;
        return SD_OK;
    };

    res->n_evaluated = 0;
    for (int32_t i = 0; i < p.n_init; ++i) {
        const sd_status rc = evaluate(initial_mask(p.seed, i, p.n_init, L), INFINITY);
        if (rc != SD_OK)
            return rc;
    }
    std::vector<double> work(cap), ei;
    std::vector<Mask> fresh;
    for (int32_t t = 0; t < p.iterations; ++t) {
        const std::vector<double> ys = standardise(y);
        gp.set_observations(ys);
        const int32_t inc = (int32_t)(std::min_element(y.begin(), y.end()) - y.begin());
        const double best = *std::min_element(ys.begin(), ys.end());
        fresh.clear();
        for (int32_t c = 0; c < p.n_candidates; ++c) {
            Mask z = candidate(p.seed, t, c, p.n_candidates, L, gp.mask(inc));
            if (!seen.count(z))
                fresh.push_back(std::move(z));
        }
        if (fresh.empty())
            continue;
        ei.resize(fresh.size());
        for (size_t c = 0; c < fresh.size(); ++c) {
            double mu, sigma;
            gp.predict(fresh[c], work.data(), &mu, &sigma);
            ei[c] = expected_improvement(mu, sigma, best, p.xi);
        }
        const size_t pick = std::max_element(ei.begin(), ei.end()) - ei.begin();
        double below = -INFINITY;
        for (double e : ei)
            if (e < ei[pick])
                below = std::max(below, e);
        const sd_status rc = evaluate(fresh[pick], ei[pick] - below);
        if (rc != SD_OK)
            return rc;
    }
    const int32_t b = (int32_t)(std::min_element(y.begin(), y.end()) - y.begin());
    std::memcpy(res->best_mask, gp.mask(b).bytes.data(), L);
    res->best_value = y[b];
    return SD_OK;
}

// The library's own decoding as the objective.
struct DecodeObjective {
    sd_model *model;
    const int32_t *prompts;
    int32_t n_prompts, prompt_len, max_new, K_max;
    float gamma;
    const sd_adaptive *adaptive;
    const sd_search_params *params;
    std::vector<int32_t> out;
};

sd_status decode_objective(const uint8_t *mask, int32_t L, void *user, double *value) {
    DecodeObjective &o = *static_cast<DecodeObjective *>(user);
    const sd_search_params &p = *o.params;
    int32_t att = 0, mlp = 0;
    for (int32_t j = 0; j < L; ++j)
        (j % 2 ? mlp : att) += mask[j] ? 0 : 1;
    double total = 0.0;
    for (int32_t i = 0; i < o.n_prompts; ++i) {
        sd_stats st{};
        const int32_t *pr = o.prompts + (size_t)i * o.prompt_len;
        const sd_status rc =
            o.adaptive ? sd_self_spec_generate_adaptive(o.model, pr, o.prompt_len, o.max_new, mask, o.K_max,
                                                        o.adaptive, o.out.data(), &st)
                       : sd_self_spec_generate(o.model, pr, o.prompt_len, o.max_new, mask, o.K_max, o.gamma,
                                               o.out.data(), &st);
        if (rc != SD_OK)
            return rc;
        if (p.objective == SD_SEARCH_MEASURED) {
            total += st.decode_ms;
        } else {
            // each operation rounded on its own, in the order written
#pragma clang fp contract(off)
            const double draft = p.cost[0] + p.cost[1] * att + p.cost[2] * mlp;
            const double nd = (double)st.n_drafted, ns = (double)st.n_stages;
            total += nd * draft + ns * p.cost[3] + p.cost[4] * (nd + ns);
        }
    }
    *value = total / ((double)o.n_prompts * o.max_new);
    return SD_OK;
}

}  // namespace

extern "C" {

sd_status sd_search_skip_set_fn(int32_t n_dims, const sd_search_params *params, sd_search_objective_fn objective,
                                void *user, sd_search_result *result) {
    try {
        sd_status rc = check_params(n_dims, params, result);
        if (rc != SD_OK)
            return rc;
        if (!objective)
            return report(SD_ERR_INVALID_ARG, "objective is null");
        return run_search(n_dims, *params, objective, user, result);
    } catch (const std::bad_alloc &) {
        return report(SD_ERR_OOM, "host allocation failed");
    } catch (...) {
        return report(SD_ERR_INVALID_ARG, "unexpected internal error");
    }
}

sd_status sd_search_skip_set(sd_model *model, const int32_t *prompts, int32_t n_prompts, int32_t prompt_len,
                             int32_t max_new, int32_t K_max, float gamma, const sd_adaptive *adaptive,
                             const sd_search_params *params, sd_search_result *result) {
    try {
        if (!model || !prompts)
            return report(SD_ERR_INVALID_ARG, "model and prompts are required");
        if (n_prompts < 1 || prompt_len < 1 || max_new < 1)
            return report(SD_ERR_INVALID_ARG, "need n_prompts, prompt_len and max_new >= 1");
        sd_status rc = check_params(2 * sdk::model_layers(model), params, result);
        if (rc != SD_OK)
            return rc;
        if (params->objective != SD_SEARCH_MEASURED && params->objective != SD_SEARCH_MODELED)
            return report(SD_ERR_INVALID_ARG, "objective must be SD_SEARCH_MEASURED or SD_SEARCH_MODELED");
        if (params->objective == SD_SEARCH_MODELED)
            for (double c : params->cost)
                if (!std::isfinite(c))
                    return report(SD_ERR_INVALID_ARG, "modeled costs must be finite");
        DecodeObjective o{model, prompts, n_prompts, prompt_len, max_new, K_max, gamma, adaptive, params,
                          std::vector<int32_t>(max_new)};
        return run_search(2 * sdk::model_layers(model), *params, decode_objective, &o, result);
    } catch (const std::bad_alloc &) {
        return report(SD_ERR_OOM, "host allocation failed");
    } catch (...) {
        return report(SD_ERR_INVALID_ARG, "unexpected internal error");
    }
}

}  // extern "C"
