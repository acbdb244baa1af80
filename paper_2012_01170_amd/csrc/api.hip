// Error reporting, tracing and small queries of the sbconv C ABI.
#include <string>
#include <unordered_map>
#include <utility>

#include "common.hpp"

namespace sbc {
namespace {
thread_local std::string g_last_error;
thread_local std::unordered_map<std::string, std::pair<hipEvent_t, hipEvent_t>> g_trace;

const char *kKernelNames =
    "points_count,points_fill,events_count,events_fill,basis,"
    "transpose_count,transpose_scatter,transpose_sort,transpose_batched,"
    "fwd_spmm,fwd_gemm,fwd_gemm_h,fwd_spmm_contract,bwd_spmm,bwd_gemm_dw,bwd_gemm_dg,"
    "bwd_spmm_t,bwd_spmm_t_expand,bwd_gemm_df,bwd_gemm_dw_t,fwd_fused,bwd_fused,bwd_dw_reduce,"
    "featureless_fwd,featureless_rowsum,featureless_dphi,decay_basis,decay_spmm,decay_gemm,"
    "decay_dot,decay_fused,decay_dw_reduce,sample_count,sample,lif_sort,lif_cells,lif_emit,stream_lists,stream_gather,stream_gemm,"
    "stream_update";
}  // namespace

void trace_before(const char *name, hipStream_t stream) {
    if (g_trace.empty()) return;
    auto it = g_trace.find(name);
    if (it != g_trace.end()) (void)hipEventRecord(it->second.first, stream);
}

void trace_after(const char *name, hipStream_t stream) {
    if (g_trace.empty()) return;
    auto it = g_trace.find(name);
    if (it != g_trace.end()) (void)hipEventRecord(it->second.second, stream);
}

void set_error(const std::string &msg) { g_last_error = msg; }

int device_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
    }
    return cus;
}
void clear_error() { g_last_error.clear(); }
sbc_status fail(sbc_status st, const std::string &msg) {
    g_last_error = msg;
    return st;
}

}  // namespace sbc

extern "C" const char *sbc_last_error(void) { return sbc::g_last_error.c_str(); }

extern "C" sbc_status sbc_trace_kernel(const char *name, hipEvent_t start, hipEvent_t stop) {
    if (!name) return sbc::fail(SBC_ERR_INVALID_ARG, "name is null");
    if (!start || !stop) {
        sbc::g_trace.erase(name);
        return SBC_OK;
    }
    sbc::g_trace[name] = {start, stop};
    return SBC_OK;
}

extern "C" void sbc_trace_clear(void) { sbc::g_trace.clear(); }

extern "C" const char *sbc_kernel_names(void) { return sbc::kKernelNames; }

extern "C" const char *sbc_status_string(sbc_status status) {
    switch (status) {
        case SBC_OK: return "ok";
        case SBC_ERR_INVALID_ARG: return "invalid argument";
        case SBC_ERR_CAPACITY: return "insufficient col_idx capacity";
        case SBC_ERR_OVERFLOW: return "edge count overflows int32";
        case SBC_ERR_UNSORTED: return "timestamps not sorted";
        case SBC_ERR_OUT_OF_RANGE: return "value out of range";
        case SBC_ERR_WORKSPACE: return "workspace too small";
        case SBC_ERR_HIP: return "HIP runtime error";
        case SBC_ERR_UNSUPPORTED: return "unsupported shape or basis";
        case SBC_ERR_INTERNAL: return "internal consistency check failed";
    }
    return "unknown status";
}

extern "C" int32_t sbc_basis_size(sbc_basis basis) {
    switch (basis) {
        case SBC_BASIS_MONO4: return 4;
        case SBC_BASIS_MONO8: return 8;
        case SBC_BASIS_EVENT8: return 8;
        case SBC_BASIS_WMONO10: return 10;
    }
    return 0;
}
