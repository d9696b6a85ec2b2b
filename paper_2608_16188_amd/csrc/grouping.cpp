// Cross-task expert grouping on the host (paper Sec. 3.2.1): the temporary
// DRAM estimate of an expert and the cut of the expert pool into ordered
// time slices, each slice the 0/1 knapsack optimum over the experts not yet
// placed (weight M_tmp in whole units, value M_tmp / M_c - eta r, capacity
// M_c - M_s). Host code only: plain pointers to host memory, no GPU work.
//
// Built without floating-point contraction: values and sums are formed by
// the operations written here, in this order, so the result is independent
// of the compiler's choice to fuse a multiply and an add.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "../../include/vmoe.h"

namespace {

constexpr int64_t kMaxUnits = int64_t(1) << 24;  // table width bound
constexpr int32_t kMaxExpertsGrouped = 1 << 16;

struct GroupPlan {
    int64_t W;       // capacity in units
    size_t bytes;    // workspace: dp row, take matrix, remaining list
    size_t take_off, rem_off;
};

bool plan_groups(int32_t n, double mem_budget, double mem_static, double unit, GroupPlan* p) {
    if (n < 0 || n > kMaxExpertsGrouped || !(unit > 0.0) || !(mem_budget > mem_static))
        return false;
    const double w = floor((mem_budget - mem_static) / unit);
    if (!(w >= 0.0) || w > static_cast<double>(kMaxUnits)) return false;
    p->W = static_cast<int64_t>(w);
    const size_t row = static_cast<size_t>(p->W) + 1;
    p->take_off = sizeof(double) * row;
    p->rem_off = p->take_off + ((static_cast<size_t>(n) * row + 7) & ~size_t(7));
    p->bytes = p->rem_off + sizeof(int32_t) * static_cast<size_t>(n);
    return true;
}

}  // namespace

extern "C" {

double vmoe_expert_mtmp(int64_t tokens, int32_t d_k, double bytes_per_elem, double theta1,
                        double theta2, double m_f) {
    const double T = static_cast<double>(tokens);
    const double m_c = bytes_per_elem * (theta1 * T * d_k + theta2 * T * T);
    return m_c + m_f;
}

size_t vmoe_group_experts_workspace_bytes(int32_t n, double mem_budget, double mem_static,
                                          double unit_bytes) {
    GroupPlan p;
    return plan_groups(n, mem_budget, mem_static, unit_bytes, &p) ? p.bytes : 0;
}

vmoe_status vmoe_group_experts(int32_t n, const double* mtmp, const double* lifespan,
                               double mem_budget, double mem_static, double eta,
                               double unit_bytes, int32_t* slice_of, int32_t* n_slices,
                               void* workspace, size_t workspace_bytes) {
    GroupPlan p;
    if (!plan_groups(n, mem_budget, mem_static, unit_bytes, &p) || !n_slices ||
        (n > 0 && (!mtmp || !lifespan || !slice_of)))
        return VMOE_ERR_INVALID_ARG;
    if (!workspace || workspace_bytes < p.bytes) return VMOE_ERR_WORKSPACE;
    const int64_t W = p.W;
    const size_t row = static_cast<size_t>(W) + 1;
    double* dp = static_cast<double*>(workspace);
    uint8_t* take = static_cast<uint8_t*>(workspace) + p.take_off;
    int32_t* rem = reinterpret_cast<int32_t*>(static_cast<uint8_t*>(workspace) + p.rem_off);
    for (int32_t i = 0; i < n; ++i) {
        if (!(mtmp[i] >= 0.0) || !(lifespan[i] >= 0.0)) return VMOE_ERR_INVALID_ARG;
        if (ceil(mtmp[i] / unit_bytes) > static_cast<double>(W)) return VMOE_ERR_INVALID_ARG;
        slice_of[i] = -1;
        rem[i] = i;
    }
    int32_t nrem = n, s = 0;
    while (nrem > 0) {
        // dp[j] = best value of the remaining experts seen so far within j
        // units; item r replaces it only when strictly better (row r of the
        // table, kept one row at a time by walking j downwards)
        for (size_t j = 0; j < row; ++j) dp[j] = 0.0;
        for (int32_t r = 0; r < nrem; ++r) {
            const int32_t i = rem[r];
            const int64_t wi = static_cast<int64_t>(ceil(mtmp[i] / unit_bytes));
            const double vi = mtmp[i] / mem_budget - eta * lifespan[i];
            uint8_t* tk = take + static_cast<size_t>(r) * row;
            memset(tk, 0, row);
            for (int64_t j = W; j >= wi; --j) {
                const double cand = dp[j - wi] + vi;
                if (cand > dp[j]) {
                    dp[j] = cand;
                    tk[j] = 1;
                }
            }
        }
        // the chosen set, read back from full capacity
        int32_t chosen = 0;
        int64_t j = W;
        for (int32_t r = nrem - 1; r >= 0; --r) {
            if (take[static_cast<size_t>(r) * row + j]) {
                const int32_t i = rem[r];
                slice_of[i] = s;
                j -= static_cast<int64_t>(ceil(mtmp[i] / unit_bytes));
                ++chosen;
            }
        }
        if (chosen == 0) {  // nothing gains: the shortest remaining job alone
            int32_t best = rem[0];
            for (int32_t r = 1; r < nrem; ++r)
                if (lifespan[rem[r]] < lifespan[best]) best = rem[r];
            slice_of[best] = s;
        }
        int32_t k = 0;
        for (int32_t r = 0; r < nrem; ++r)
            if (slice_of[rem[r]] < 0) rem[k++] = rem[r];
        nrem = k;
        ++s;
    }
    *n_slices = s;
    return VMOE_OK;
}

// Fill-clamp-refill allocation of compute units within a slice (paper
// Sec. 3.2.2): minima first, the rest in proportion to the coefficients among
// the unsaturated experts, saturated experts clamped and their excess shared
// again, until nothing is returned. Real shares in `alloc`, their
// largest-remainder rounding to floor(sum) whole units in `alloc_units`
// (ties to the lower index); `n_rounds` counts the share-clamp rounds.
vmoe_status vmoe_fill_clamp_refill(int32_t n, const int32_t* min_units, const int32_t* sat_units,
                                   const double* coef, int64_t budget, double* alloc,
                                   int32_t* alloc_units, int32_t* n_rounds, void* workspace,
                                   size_t workspace_bytes) {
    if (n < 0 || n > kMaxExpertsGrouped || !n_rounds ||
        (n > 0 && (!min_units || !sat_units || !coef || !alloc || !alloc_units)))
        return VMOE_ERR_INVALID_ARG;
    if (workspace_bytes < sizeof(int32_t) * static_cast<size_t>(n) || (n > 0 && !workspace))
        return VMOE_ERR_WORKSPACE;
    int64_t need = 0;
    for (int32_t i = 0; i < n; ++i) {
        if (min_units[i] < 0 || sat_units[i] < min_units[i] || !(coef[i] >= 0.0) ||
            !isfinite(coef[i]))
            return VMOE_ERR_INVALID_ARG;
        need += min_units[i];
    }
    if (budget < need) return VMOE_ERR_INVALID_ARG;
    int32_t* active = static_cast<int32_t*>(workspace);
    int32_t na = 0;
    for (int32_t i = 0; i < n; ++i) {
        alloc[i] = static_cast<double>(min_units[i]);
        if (alloc[i] < sat_units[i] && coef[i] > 0.0) active[na++] = i;
    }
    double left = static_cast<double>(budget - need);
    int32_t rounds = 0;
    while (left > 0.0 && na > 0) {
        double W = 0.0;
        for (int32_t r = 0; r < na; ++r) W += coef[active[r]];
        for (int32_t r = 0; r < na; ++r) alloc[active[r]] += left * coef[active[r]] / W;
        ++rounds;
        left = 0.0;
        int32_t kept = 0;
        for (int32_t r = 0; r < na; ++r) {
            const int32_t i = active[r];
            if (alloc[i] > sat_units[i]) {
                left += alloc[i] - sat_units[i];
                alloc[i] = static_cast<double>(sat_units[i]);
            } else {
                active[kept++] = i;
            }
        }
        na = kept;
    }
    // whole units: floor of each share, then the remaining units to the
    // largest fractional parts (lower index first on ties)
    double sum = 0.0;
    int64_t base = 0;
    for (int32_t i = 0; i < n; ++i) {
        alloc_units[i] = static_cast<int32_t>(floor(alloc[i]));
        base += alloc_units[i];
        sum += alloc[i];
    }
    int64_t extra = static_cast<int64_t>(floor(sum + 1e-9)) - base;
    while (extra > 0) {
        int32_t best = -1;
        double bf = 0.0;  // only shares with a fractional part round up
        for (int32_t i = 0; i < n; ++i) {
            const double fr = alloc[i] - floor(alloc[i]);
            if (alloc_units[i] == static_cast<int32_t>(floor(alloc[i])) && fr > bf) {
                best = i;
                bf = fr;
            }
        }
        if (best < 0) break;
        ++alloc_units[best];
        --extra;
    }
    *n_rounds = rounds;
    return VMOE_OK;
}

}  // extern "C"
