// cells.hip -- C ABI of GPipe's cell partitioner (host code; see cells.hpp).
#include <string>

#include "cells.hpp"

namespace gp {
gp_status set_error(gp_status s, const char* msg);
}

extern "C" gp_status gp_plan_cells(const double* costs, int layers, int cells, int* first_layer, double* variance) {
    std::string msg;
    const gp_status s = gp::plan_cells(costs, layers, cells, first_layer, variance, msg);
    if (s != GP_OK) return gp::set_error(s, msg.c_str());
    return GP_OK;
}
