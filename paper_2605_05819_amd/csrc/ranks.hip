// Compensation-rank allocation from the residual spectra (Section 4.3.1 and
// 4.3.4; Appendix B.1).  Host code only: it turns the singular values that
// cl_build_compensation writes, plus sensitivity scores, into the per-linear
// ranks the decode and prefill entry points take.  Every sum runs in index
// order in fp64, so a result does not depend on the build.

#include <math.h>

#include "cl_internal.h"

namespace cl {

namespace {

// Proportional shares of `budget` over items with weights w and caps cap,
// water-filling: each round gives every open item (positive weight, room
// left) its weight's share of what is left; if a share would pass an item's
// cap, the item is filled to its cap instead and closed, and the round's
// other shares are not given.  Ends when a round closes nothing or nothing
// is left.
void waterfill(int n, const double* w, const double* cap, double budget, double* out) {
    bool open[kMaxRankWin];
    for (int i = 0; i < n; ++i) {
        out[i] = 0.0;
        open[i] = w[i] > 0.0 && cap[i] > 0.0;
    }
    double left = budget;
    while (left > 0.0) {
        double wsum = 0.0;
        for (int i = 0; i < n; ++i)
            if (open[i]) wsum += w[i];
        if (!(wsum > 0.0)) break;
        bool closed = false;
        for (int i = 0; i < n; ++i) {
            if (!open[i]) continue;
            const double room = cap[i] - out[i];
            if (left * w[i] / wsum >= room) {
                out[i] = cap[i];
                open[i] = false;
                closed = true;
            }
        }
        if (closed) {
            double used = 0.0;
            for (int i = 0; i < n; ++i) used += out[i];
            left = budget - used;
            continue;
        }
        for (int i = 0; i < n; ++i)
            if (open[i]) out[i] += left * w[i] / wsum;
        break;
    }
}

}  // namespace

int salient_count(const float* sigma, int n, double tau, double* phi) {
    *phi = 1.0;
    if (n < 3 || !(sigma[0] > 0.0f)) return 0;
    const double s1 = sigma[0];
    // second differences of sigma / sigma_1 at the interior indices; the
    // first largest one marks the end of the salient set
    double best = -INFINITY;
    int at = 0;
    for (int j = 1; j + 1 < n; ++j) {
        const double k = sigma[j - 1] / s1 - 2.0 * (sigma[j] / s1) + sigma[j + 1] / s1;
        if (k > best) {
            best = k;
            at = j;
        }
    }
    if (!(best > tau)) return 0;
    const int cnt = at + 1;
    double ssum = 0.0, rsum = 0.0;
    for (int j = 0; j < cnt; ++j) ssum += sigma[j];
    for (int j = cnt; j < n; ++j) rsum += sigma[j];
    const double smean = ssum / cnt, rmean = rsum / (n - cnt);
    *phi = rmean > 0.0 ? smean / rmean : INFINITY;
    return cnt;
}

void allocate_window_ranks(int n, const float* const* sigma, const int* len, const double* sens, double layer_score,
                           double r_std, const int* levels, int nlevels, int r_max, double tau, int* ranks,
                           double* cont) {
    double phi[kMaxRankWin], v[kMaxRankWin], s[kMaxRankWin], x[kMaxRankWin], rt[kMaxRankWin];
    double sal[kMaxRankWin], res[kMaxRankWin], a[kMaxRankWin], b[kMaxRankWin];
    // recoverability: salience ratios normalised over the window; an infinite
    // ratio (a residual set of zeros) takes the whole share, split evenly
    int ninf = 0;
    double psum = 0.0;
    for (int i = 0; i < n; ++i) {
        const int c = salient_count(sigma[i], len[i], tau, &phi[i]);
        sal[i] = c;
        res[i] = len[i] - c;
        if (isinf(phi[i])) ++ninf;
        else psum += phi[i];
    }
    for (int i = 0; i < n; ++i)
        v[i] = ninf ? (isinf(phi[i]) ? 1.0 / ninf : 0.0) : phi[i] / psum;
    // matrix-level sensitivity normalised over the window (all zero: even)
    double dsum = 0.0;
    for (int i = 0; i < n; ++i) dsum += sens[i];
    for (int i = 0; i < n; ++i) s[i] = dsum > 0.0 ? sens[i] / dsum : 1.0 / n;
    // priority: the normalised product times the layer score; continuous rank
    double xsum = 0.0;
    for (int i = 0; i < n; ++i) {
        x[i] = v[i] * s[i];
        xsum += x[i];
    }
    double budget = 0.0;
    for (int i = 0; i < n; ++i) {
        const double p = xsum > 0.0 ? x[i] / xsum * layer_score : 0.0;
        rt[i] = p * r_std;
        budget += rt[i];
    }
    // two stages: the budget goes to the salient sets first, the rest to the
    // residual sets, both in proportion to the continuous ranks
    waterfill(n, rt, sal, budget, a);
    double used = 0.0;
    for (int i = 0; i < n; ++i) used += a[i];
    waterfill(n, rt, res, budget - used, b);
    for (int i = 0; i < n; ++i) {
        const double c = a[i] + b[i];
        if (cont) cont[i] = c;
        // nearest admissible level within min(r_max, len), ties to the lower
        const int top = len[i] < r_max ? len[i] : r_max;
        int r = levels[0];
        for (int l = 1; l < nlevels && levels[l] <= top; ++l)
            if (fabs(c - levels[l]) < fabs(c - r)) r = levels[l];
        ranks[i] = r;
    }
}

void layer_sensitivity(int L, const double* D, int K, double* S) {
    // top-K layers by D (ties to the lower index) score 1; the others D over
    // the smallest D among the top K (0 / 0 reads as 1)
    bool top[kMaxLayers];
    for (int l = 0; l < L; ++l) top[l] = false;
    double dmin = INFINITY;
    for (int k = 0; k < K; ++k) {
        int best = -1;
        for (int l = 0; l < L; ++l)
            if (!top[l] && (best < 0 || D[l] > D[best])) best = l;
        top[best] = true;
        if (D[best] < dmin) dmin = D[best];
    }
    for (int l = 0; l < L; ++l) S[l] = top[l] ? 1.0 : (dmin > 0.0 ? D[l] / dmin : 1.0);
}

}  // namespace cl
