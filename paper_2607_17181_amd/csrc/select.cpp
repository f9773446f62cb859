// SP batch selection (host), after Section 3.4: at each SP opportunity a
// bounded set of the waiting returning continuations is taken, sized so that
// its predicted cost (attention time, page restore time, device pages) stays
// inside what the slot has left once decode is served; the others wait for
// a later opportunity.
//
// Rule: candidates are taken in queue (arrival) order; each is admitted if
// the batch with it still fits every bound -- predicted time, free device
// pages and batch size -- and is otherwise skipped and left queued, and the
// scan continues with the next (first fit).
//
// A host-resident prefix is restored page-aligned (only whole pages are
// agreed and checkpointed, Appendix B); its partial last page is recomputed
// with the suffix, so such a candidate enters the batch with prefix
// P' = floor(P / ps) * ps and suffix S' = S + P - P'.  Costs per candidate
// (with these effective lengths):
//   attention FLOPs = 4 d Hq layers (S P + S (S+1) / 2)
//   T_pf      = FLOPs / attn_flops_per_s + S * per_token_s
//   T_restore = (host-resident) P' / ps pages * K+V page bytes of all layers
//               / restore_bytes_per_s, else 0
//   pages     = device pages the batch must allocate: the suffix's pages past
//               the prefix's last page, or every page when the prefix is
//               restored into new slots
// and one batch_overhead_s per non-empty batch.
#include <hip/hip_runtime.h>

#include <math.h>

#include "common.h"

using namespace tsp;

namespace {

struct CandCost {
    double seconds;
    int64_t pages;
    int32_t prefix, suffix;  // lengths the batch's plan uses
};

CandCost candidate_cost(const talaria_sp_candidate& c, const talaria_sp_cost_model& m) {
    const int64_t ps = m.page_size;
    int32_t P = c.prefix_len, S = c.suffix_len;
    if (c.host_resident) {
        const int32_t aligned = (int32_t)((P / ps) * ps);
        S += P - aligned;
        P = aligned;
    }
    const double Pd = P, Sd = S;
    const double flops = 4.0 * m.head_dim * m.num_q_heads * (double)m.num_layers *
                         (Sd * Pd + Sd * (Sd + 1.0) / 2.0);
    double t = flops / m.attn_flops_per_s + Sd * m.per_token_s;
    const int64_t total_pages = ((int64_t)P + S + ps - 1) / ps;
    int64_t pages;
    if (c.host_resident) {
        const double page_bytes = 2.0 * m.num_kv_heads * ps * m.head_dim * 2.0 * m.num_layers;
        t += (double)(P / ps) * page_bytes / m.restore_bytes_per_s;
        pages = total_pages;
    } else {
        pages = total_pages - ((int64_t)P + ps - 1) / ps;
    }
    return {t, pages, P, S};
}

}  // namespace

extern "C" int talaria_sp_select(const talaria_sp_candidate* cands, int32_t num_cands,
                                 const talaria_sp_cost_model* model,
                                 const talaria_sp_budget* budget, int32_t* selected,
                                 int32_t* plan_prefix_lens, int32_t* plan_suffix_lens,
                                 double* predicted_seconds, int64_t* predicted_pages) {
    if (num_cands < 0 || !model || !budget || (num_cands > 0 && (!cands || !selected)))
        return fail(TALARIA_SP_EINVAL, "sp_select: bad arguments");
    const talaria_sp_cost_model& m = *model;
    if (m.num_layers <= 0 || m.num_q_heads <= 0 || m.num_kv_heads <= 0 || m.head_dim <= 0 ||
        m.page_size <= 0 || !(m.attn_flops_per_s > 0) || !isfinite(m.attn_flops_per_s) ||
        !(m.restore_bytes_per_s > 0) || !isfinite(m.restore_bytes_per_s) ||
        !(m.per_token_s >= 0) || !isfinite(m.per_token_s) || !(m.batch_overhead_s >= 0) ||
        !isfinite(m.batch_overhead_s) || isnan(budget->time_budget_s))
        return fail(TALARIA_SP_EINVAL, "sp_select: cost model must be positive and finite");
    if (budget->max_batch < 0 || budget->max_batch > TALARIA_SP_MAX_SEQS)
        return fail(TALARIA_SP_EINVAL, "sp_select: max_batch must be in [0, %d]",
                    TALARIA_SP_MAX_SEQS);
    double t = 0.0;
    int64_t pages = 0;
    int32_t n = 0;
    for (int32_t i = 0; i < num_cands && n < budget->max_batch; ++i) {
        const talaria_sp_candidate& c = cands[i];
        if (c.prefix_len < 0 || c.suffix_len <= 0)
            continue;  // nothing to prefill
        const CandCost k = candidate_cost(c, m);
        const double t_new = t + k.seconds + (n == 0 ? m.batch_overhead_s : 0.0);
        const int64_t p_new = pages + k.pages;
        if (t_new <= budget->time_budget_s && p_new <= budget->free_pages) {
            t = t_new;
            pages = p_new;
            if (plan_prefix_lens)
                plan_prefix_lens[n] = k.prefix;
            if (plan_suffix_lens)
                plan_suffix_lens[n] = k.suffix;
            selected[n++] = i;
        }
    }
    if (predicted_seconds)
        *predicted_seconds = t;
    if (predicted_pages)
        *predicted_pages = pages;
    return n;
}
