// Threshold calibration helpers (App. A.7): each layer keeps a bounded
// sample of every calibration signal, and a threshold is the empirical
// quantile of that sample at the target sparsity.  Host code only: these run
// offline, between the GPU forward passes that produce the samples.
#include <prox.h>

#include <algorithm>
#include <cmath>
#include <vector>

extern "C" {

prox_status prox_reservoir_add(float *reservoir, size_t cap, uint64_t *seen, const float *values,
                               size_t n, const uint64_t *draws) {
    if (!reservoir || !seen || cap == 0 || (n && (!values || !draws))) return PROX_ERR_INVALID;
    // Algorithm R: offer number t fills slot t while the reservoir has room,
    // then takes slot (draw mod (t + 1)) when that slot exists.
    for (size_t i = 0; i < n; ++i) {
        const uint64_t t = *seen + i;
        if (t < cap) {
            reservoir[t] = values[i];
        } else {
            const uint64_t slot = draws[i] % (t + 1);
            if (slot < cap) reservoir[slot] = values[i];
        }
    }
    *seen += n;
    return PROX_OK;
}

prox_status prox_quantile_threshold(const float *samples, size_t n, double sparsity,
                                    float *tau) {
    if (!samples || !tau || n == 0 || !(sparsity >= 0.0 && sparsity < 1.0))
        return PROX_ERR_INVALID;
    std::vector<float> v(samples, samples + n);
    for (float s : v)
        if (std::isnan(s)) return PROX_ERR_INVALID;
    size_t pos = (size_t)std::floor(sparsity * (double)n);
    if (pos > n - 1) pos = n - 1;
    std::nth_element(v.begin(), v.begin() + (std::ptrdiff_t)pos, v.end());
    *tau = v[pos];   // the pos-th smallest: about sparsity * n samples lie below it
    return PROX_OK;
}

// Sec. 4.2 cost model: a dense projection costs 1 and a proxy projection
// alpha; Stage 1 runs two proxy projections over the kept (1 - s1) inputs,
// Stage 2 three exact ones over the kept (1 - s2) channels.
double prox_effective_sparsity(double s1, double s2, double alpha) {
    const double cost = 2.0 * alpha * (1.0 - s1) + 3.0 * (1.0 - s2);
    return 1.0 - cost / 3.0;   // against the dense cost of 3
}

prox_status prox_allocate_sparsity(double e, double alpha, double s_ref, double s1_min,
                                   double s1_max, double *s1, double *s2) {
    if (!s1 || !s2 || !(alpha > 0.0) || !(s1_min <= s1_max) || std::isnan(e) ||
        std::isnan(s_ref) || std::isnan(s1_min) || std::isnan(s1_max))
        return PROX_ERR_INVALID;
    // Stage 2 at its anchor, Stage 1 takes the rest of the budget; a Stage 1
    // share outside its bounds is clamped and Stage 2 solved again.
    double b = s_ref;
    double a = 1.0 - 1.5 * (b - e) / alpha;
    if (a < s1_min || a > s1_max) {
        a = std::min(std::max(a, s1_min), s1_max);
        b = e + 2.0 * alpha * (1.0 - a) / 3.0;
    }
    *s1 = a;
    *s2 = b;
    return PROX_OK;
}

}  // extern "C"
