// controller.cpp -- adaptive speculation length (Sec. 3.3), host only.
//
// Tracks the mean draft entropy of accepted and of rejected tokens with
// exponential moving averages (Eq. 6), turns a new draft's entropy into a soft
// acceptance probability by its closeness to the two class means (Eq. 7), and
// picks the candidate speculation length with the most expected tokens per
// unit of step cost (Eq. 8).
#include <math.h>

#include <algorithm>
#include <new>
#include <vector>

#include "../../include/sparsespec_l.h"

struct ssl_ctrl {
    double beta;
    std::vector<int32_t> cands;
    int32_t k_default;
    double h_acc, h_rej;
    bool seen_acc, seen_rej;
};

namespace {

double class_mean(const double* H, int32_t lo, int32_t hi) {
    double s = 0.0;
    for (int32_t i = lo; i < hi; ++i) s += H[i];
    return s / (double)(hi - lo);
}

// Eq. 7 written as 1 / (1 + e^(d_acc - d_rej)): the printed ratio of
// exponentials divided through by its numerator, so that large distances do
// not underflow both terms.
double accept_prob(const ssl_ctrl* c, double H) {
    if (!c->seen_acc || !c->seen_rej) return 0.5;
    const double d_acc = fabs(H - c->h_acc);
    const double d_rej = fabs(H - c->h_rej);
    return 1.0 / (1.0 + exp(d_acc - d_rej));
}

}  // namespace

extern "C" {

ssl_ctrl* ssl_ctrl_create(double beta, const int32_t* k_cands, int32_t n_cands, int32_t k_default) {
    if (!(beta >= 0.0 && beta <= 1.0) || !k_cands || n_cands < 1 || n_cands > 256) return nullptr;
    for (int32_t i = 0; i < n_cands; ++i)
        if (k_cands[i] < 0) return nullptr;
    ssl_ctrl* c = new (std::nothrow) ssl_ctrl;
    if (!c) return nullptr;
    c->beta = beta;
    c->cands.assign(k_cands, k_cands + n_cands);
    c->k_default = k_default;
    c->h_acc = c->h_rej = 0.0;
    c->seen_acc = c->seen_rej = false;
    return c;
}

void ssl_ctrl_destroy(ssl_ctrl* c) { delete c; }

int ssl_ctrl_observe(ssl_ctrl* c, const double* H, int32_t n_drafted, int32_t n_accepted) {
    if (!c || (n_drafted > 0 && !H)) return SSL_ERR_NULL;
    if (n_drafted < 0 || n_accepted < 0 || n_accepted > n_drafted) return SSL_ERR_SHAPE;
    if (n_accepted > 0) {
        const double m = class_mean(H, 0, n_accepted);
        c->h_acc = c->seen_acc ? c->beta * c->h_acc + (1.0 - c->beta) * m : m;
        c->seen_acc = true;
    }
    if (n_drafted > n_accepted) {
        const double m = class_mean(H, n_accepted, n_drafted);
        c->h_rej = c->seen_rej ? c->beta * c->h_rej + (1.0 - c->beta) * m : m;
        c->seen_rej = true;
    }
    return SSL_OK;
}

double ssl_ctrl_accept_prob(const ssl_ctrl* c, double H) {
    if (!c) return NAN;
    return accept_prob(c, H);
}

int32_t ssl_ctrl_choose_k(const ssl_ctrl* c, const double* H, int32_t n, double c_draft,
                          double c_verify) {
    if (!c || (n > 0 && !H)) return SSL_ERR_NULL;
    if (n < 0) return SSL_ERR_SHAPE;
    // Eq. 8 divides by k * c_draft + c_verify
    if (!isfinite(c_draft) || !isfinite(c_verify) || c_draft < 0.0 || !(c_verify > 0.0))
        return SSL_ERR_SHAPE;
    if (!c->seen_acc || !c->seen_rej) return c->k_default;
    // Prefix sums of the acceptance-prefix probabilities, then one pass over
    // the candidates.
    std::vector<double> cum((size_t)n + 1, 0.0);
    double prod = 1.0;
    for (int32_t m = 1; m <= n; ++m) {
        prod *= accept_prob(c, H[m - 1]);
        cum[m] = cum[m - 1] + prod;
    }
    int32_t best = -1;
    double best_val = 0.0;
    for (int32_t k : c->cands) {
        if (k > n) continue;
        const double val = (1.0 + cum[k]) / ((double)k * c_draft + c_verify);
        if (best < 0 || val > best_val || (val == best_val && k < best)) {
            best = k;
            best_val = val;
        }
    }
    return best < 0 ? SSL_ERR_SHAPE : best;
}

int ssl_ctrl_get_state(const ssl_ctrl* c, double* out4) {
    if (!c || !out4) return SSL_ERR_NULL;
    out4[0] = c->h_acc;
    out4[1] = c->h_rej;
    out4[2] = c->seen_acc ? 1.0 : 0.0;
    out4[3] = c->seen_rej ? 1.0 : 0.0;
    return SSL_OK;
}

int ssl_ctrl_set_state(ssl_ctrl* c, const double* in4) {
    if (!c || !in4) return SSL_ERR_NULL;
    c->h_acc = in4[0];
    c->h_rej = in4[1];
    c->seen_acc = in4[2] != 0.0;
    c->seen_rej = in4[3] != 0.0;
    return SSL_OK;
}

}  // extern "C"
