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

}  // extern "C"
