// cells.hpp -- GPipe's partitioning of a layer sequence into K cells
// (HIP-free host code; unit-tested without a GPU).
//
// Each layer i carries a cost estimate c_i, and a cell of consecutive layers
// i..j costs C_k = c_i + ... + c_j (Section 2.1).  The split into K cells
// minimises the variance of the cell costs (Section 2.2).  With the mean
// (sum of all c_i) / K fixed, the variance (1/K) sum_k C_k^2 - mean^2 is least
// where sum_k C_k^2 is, which a dynamic program over prefix sums finds
// exactly: best[k][j] = min over i < j of best[k-1][i] + (P_j - P_i)^2, the
// least sum of squares of k cells covering layers 0..j-1, O(K L^2) time and
// O(K L) memory.  Ties keep the smallest cut, so the split is deterministic.
#pragma once

#include <cmath>
#include <limits>
#include <string>
#include <vector>

#include "../../include/gp.h"

namespace gp {

inline gp_status plan_cells(const double* costs, int L, int K, int* first, double* var, std::string& msg) {
    if (!costs || !first) {
        msg = "costs and first_layer must not be NULL";
        return GP_ERR_INVALID_ARG;
    }
    if (L < 1 || K < 1 || K > L) {
        msg = "need 1 <= cells <= layers";
        return GP_ERR_INVALID_ARG;
    }
    std::vector<double> P(L + 1, 0.0);
    for (int i = 0; i < L; ++i) {
        if (!std::isfinite(costs[i]) || costs[i] < 0.0) {
            msg = "layer costs must be finite and non-negative";
            return GP_ERR_INVALID_ARG;
        }
        P[i + 1] = P[i] + costs[i];
    }
    const double inf = std::numeric_limits<double>::infinity();
    // best[k][j]: k + 1 cells over layers 0..j-1; from[k][j]: first layer of the last of them
    std::vector<std::vector<double>> best(K, std::vector<double>(L + 1, inf));
    std::vector<std::vector<int>> from(K, std::vector<int>(L + 1, -1));
    for (int j = 1; j <= L; ++j) {
        best[0][j] = P[j] * P[j];
        from[0][j] = 0;
    }
    for (int k = 1; k < K; ++k) {
        for (int j = k + 1; j <= L; ++j) {
            for (int i = k; i < j; ++i) {
                const double c = P[j] - P[i];
                const double v = best[k - 1][i] + c * c;
                if (v < best[k][j]) {
                    best[k][j] = v;
                    from[k][j] = i;
                }
            }
        }
    }
    int j = L;
    for (int k = K - 1; k >= 0; --k) {
        first[k] = from[k][j];
        j = first[k];
    }
    if (var) {
        const double mean = P[L] / K;
        double s = 0.0;
        for (int k = 0; k < K; ++k) {
            const double c = P[k + 1 < K ? first[k + 1] : L] - P[first[k]] - mean;
            s += c * c;
        }
        *var = s / K;
    }
    return GP_OK;
}

} // namespace gp
