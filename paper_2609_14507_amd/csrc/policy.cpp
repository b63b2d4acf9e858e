// Roofline CPU/GPU split policy (Sec. 5.2-5.3): host-side scheduling that
// decides how much of each sequence the CPU partition takes.  Plain C++, no
// GPU work.
//
//   Eq. 1   T_cpu(r) = r A L + C_cpu,   T_gpu(r) = (1 - r) B L + C_gpu
//   Eq. 2   r(L) = clamp(B/(A+B) + (C_gpu - C_cpu)/((A+B) L), 0, 1)
//
// Decode evictions are routed batch by batch so that the running fraction of
// CPU-placed batches follows the marginal share p = B/(A+B); A drifts with
// the workload and is re-estimated from a sliding window of measured CPU
// latencies.

// Contraction to fused multiply-adds stays off: the decisions must equal those
// of a plain evaluation of the formulas.
#pragma clang fp contract(off)

#include <cmath>
#include <cstdlib>
#include <new>
#include <vector>

#include "wsk.h"
#include "wsk_internal.h"

namespace {

bool valid_model(const wsk_roofline *m) {
    return m && std::isfinite(m->A) && std::isfinite(m->B) && std::isfinite(m->c_cpu) &&
           std::isfinite(m->c_gpu) && m->A >= 0.0 && m->B >= 0.0 && m->A + m->B > 0.0 && m->c_cpu >= 0.0 &&
           m->c_gpu >= 0.0;
}

double share_of(const wsk_roofline &m, double L) {
    const double delta = m.c_gpu - m.c_cpu;
    const double x = m.B / (m.A + m.B) + delta / ((m.A + m.B) * L);
    return x > 1.0 ? 1.0 : (x < 0.0 ? 0.0 : x);
}

}  // namespace

struct wsk_policy {
    wsk_roofline m;
    int32_t window = 1;
    std::vector<double> t;       // ring of the last `window` CPU latencies
    std::vector<int64_t> n;      // and CPU token counts
    int32_t filled = 0, next = 0;
    int64_t batches = 0, cpu_batches = 0;
};

extern "C" {

int wsk_roofline_share(const wsk_roofline *m, int64_t L, double *r) {
    if (!valid_model(m) || L < 1 || !r) return wsk::policy_fail(WSK_EINVAL, "roofline model or L");
    *r = share_of(*m, (double)L);
    return WSK_OK;
}

int wsk_policy_create(const wsk_roofline *m0, int32_t window, wsk_policy **out) {
    if (!out) return wsk::policy_fail(WSK_EINVAL, "out is NULL");
    *out = nullptr;
    if (!valid_model(m0) || m0->A <= 0.0 || window < 1)
        return wsk::policy_fail(WSK_EINVAL, "policy needs A > 0, B >= 0 and window >= 1");
    wsk_policy *p = new (std::nothrow) wsk_policy();
    if (!p) return wsk::policy_fail(WSK_ENOMEM, "host allocation failed");
    p->m = *m0;
    p->window = window;
    p->t.assign(window, 0.0);
    p->n.assign(window, 0);
    *out = p;
    return WSK_OK;
}

int wsk_policy_destroy(wsk_policy *p) {
    delete p;
    return WSK_OK;
}

int wsk_policy_observe(wsk_policy *p, double t_cpu, int64_t n_cpu, double *A) {
    if (!p || !std::isfinite(t_cpu) || t_cpu < 0.0 || n_cpu < 0)
        return wsk::policy_fail(WSK_EINVAL, "observation");
    p->t[p->next] = t_cpu;
    p->n[p->next] = n_cpu;
    p->next = (p->next + 1) % p->window;
    if (p->filled < p->window) ++p->filled;
    // sums in the order the samples arrived (oldest first)
    double st = 0.0;
    int64_t sn = 0;
    const int first = (p->next - p->filled + p->window) % p->window;
    for (int k = 0; k < p->filled; ++k) {
        const int j = (first + k) % p->window;
        st += p->t[j];
        sn += p->n[j];
    }
    if (sn > 0) {
        const double a = (st - p->filled * p->m.c_cpu) / (double)sn;
        if (a > 0.0) p->m.A = a;
    }
    if (A) *A = p->m.A;
    return WSK_OK;
}

int wsk_policy_model(const wsk_policy *p, wsk_roofline *m) {
    if (!p || !m) return wsk::policy_fail(WSK_EINVAL, "NULL argument");
    *m = p->m;
    return WSK_OK;
}

int wsk_policy_route_batch(wsk_policy *p, int32_t *part) {
    if (!p || !part) return wsk::policy_fail(WSK_EINVAL, "NULL argument");
    const double share = p->m.B / (p->m.A + p->m.B);
    const bool to_cpu = (double)p->cpu_batches + 0.5 < share * (double)(p->batches + 1);
    ++p->batches;
    if (to_cpu) ++p->cpu_batches;
    *part = to_cpu ? WSK_PART_CPU : WSK_PART_GPU;
    return WSK_OK;
}

}  // extern "C"
