// Host argument checks of the C ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer (built by tests/test_sanitize.py, host code
// instrumented, no GPU needed).  Every call here is rejected (or is a size
// query) before anything is enqueued, so no kernel runs; the pointers are
// fake and never dereferenced.  Exits non-zero on the first unexpected
// status; a sanitizer report aborts the run.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "mp.h"
#include "mp_probe.h"

namespace {
int failures = 0;
void expect(const char* what, int got, int want) {
    if (got != want) {
        std::fprintf(stderr, "%s: status %d, expected %d\n", what, got, want);
        ++failures;
    }
}
void* const F = reinterpret_cast<void*>(uintptr_t(0x10000));
template <typename T>
T* fk(uintptr_t off = 0) { return reinterpret_cast<T*>(uintptr_t(0x10000) + off); }
}  // namespace

int main() {
    expect("version", mp_version(), MP_VERSION);
    for (int st = -10; st <= 0; ++st)
        if (!mp_status_str(st) || !std::strcmp(mp_status_str(st), "unknown status")) ++failures;
    if (std::strcmp(mp_status_str(-99), "unknown status")) ++failures;

    // size queries
    size_t b = 0;
    expect("csr ws", mp_coo_to_csr_workspace(1000, 50, MP_I32, 1, &b), MP_OK);
    expect("csr ws E<0", mp_coo_to_csr_workspace(-1, 50, MP_I32, 0, &b), MP_ERR_SIZE);
    expect("csr ws N=0", mp_coo_to_csr_workspace(5, 0, MP_I32, 0, &b), MP_ERR_SIZE);
    expect("csr ws itype", mp_coo_to_csr_workspace(5, 5, 7, 0, &b), MP_ERR_DTYPE);
    expect("csr ws null", mp_coo_to_csr_workspace(5, 5, MP_I32, 0, nullptr), MP_ERR_NULL);
    expect("plan size", mp_spmm_plan_size(3000, 40000, &b), MP_OK);
    expect("plan size big", mp_spmm_plan_size(int64_t(1) << 32, 1, &b), MP_ERR_SIZE);
    expect("spmm ws", mp_spmm_workspace(nullptr, MP_SUM | MP_MAX, &b), MP_OK);
    expect("spmm ws reduce", mp_spmm_workspace(nullptr, MP_SUM | MP_MEAN, &b), MP_ERR_REDUCE);
    expect("multi ws", mp_spmm_multi_workspace(nullptr, &b), MP_OK);
    expect("transpose ws", mp_csr_transpose_workspace(1000, 50, MP_I64, 1, &b), MP_OK);
    expect("bwx ws", mp_spmm_backward_x_workspace(nullptr, 10, 1000, 100, MP_MAX, &b), MP_OK);
    expect("bwx ws reduce", mp_spmm_backward_x_workspace(nullptr, 10, 10, 8, 3, &b), MP_ERR_REDUCE);
    expect("bww ws", mp_spmm_backward_w_workspace(1000, &b), MP_OK);
    expect("msg bw ws", mp_message_backward_workspace(1000, &b), MP_OK);
    expect("gmm ws", mp_segment_matmul_workspace(3, 128, 64, &b), MP_OK);
    int64_t seg[4] = {0, 100, 100, 5000};
    expect("gmm bw ws", mp_segment_matmul_backward_workspace(seg, 3, 128, 64, &b), MP_OK);
    int64_t bad_seg[3] = {0, 10, 5};
    expect("gmm bw ws seg", mp_segment_matmul_backward_workspace(bad_seg, 2, 128, 64, &b),
           MP_ERR_SIZE);
    int64_t npt[2] = {10, 5};
    mp_relation rel{0, 1, fk<int32_t>(), fk<int32_t>(), 20};
    expect("hetero ws", mp_hetero_build_workspace(2, npt, 1, &rel, 1, MP_I32, &b), MP_OK);
    expect("hetero ws all", mp_hetero_build_workspace(2, npt, 1, &rel, MP_ALL_TYPES, MP_I32, &b),
           MP_OK);
    expect("hetero ws type", mp_hetero_build_workspace(2, npt, 1, &rel, 2, MP_I32, &b), MP_ERR_SIZE);

    // COO -> CSR and the sorted fast path
    expect("csr itype", mp_coo_to_csr(fk<int32_t>(), fk<int32_t>(), 10, 5, F, 7, fk<int32_t>(),
                                      nullptr, nullptr, nullptr, F, 1 << 20, nullptr, nullptr),
           MP_ERR_DTYPE);
    expect("csr null", mp_coo_to_csr(nullptr, fk<int32_t>(), 10, 5, F, MP_I32, fk<int32_t>(),
                                     nullptr, nullptr, nullptr, F, 1 << 20, nullptr, nullptr),
           MP_ERR_NULL);
    expect("csr align", mp_coo_to_csr(fk<int32_t>(), fk<int32_t>(), 10, 5, fk<char>(4), MP_I64,
                                      fk<int32_t>(), nullptr, nullptr, nullptr, F, 1 << 20,
                                      nullptr, nullptr),
           MP_ERR_ALIGN);
    expect("csr status align", mp_coo_to_csr(fk<int32_t>(), fk<int32_t>(), 10, 5, F, MP_I32,
                                             fk<int32_t>(), nullptr, nullptr, nullptr, F, 1 << 20,
                                             fk<int32_t>(2), nullptr),
           MP_ERR_ALIGN);
    expect("csr ws small", mp_coo_to_csr(fk<int32_t>(), fk<int32_t>(), 10, 5, F, MP_I32,
                                         fk<int32_t>(), nullptr, nullptr, nullptr, F, 16, nullptr,
                                         nullptr),
           MP_ERR_WORKSPACE);
    expect("sorted itype", mp_sorted_coo_to_csr(fk<int32_t>(), fk<int32_t>(), 10, 5, F, 7,
                                                fk<int32_t>(), nullptr, nullptr, nullptr, nullptr),
           MP_ERR_DTYPE);

    // plan
    mp_plan* h = nullptr;
    expect("plan ws", mp_spmm_plan_build(F, MP_I32, 100, 1000, 64, MP_F32, F, 16, nullptr, &h),
           MP_ERR_WORKSPACE);
    expect("plan F", mp_spmm_plan_build(F, MP_I32, 100, 1000, 0, MP_F32, F, 1 << 30, nullptr, &h),
           MP_ERR_SIZE);
    mp_plan_opts o{-1, 0, 0};
    expect("plan opts", mp_spmm_plan_build_opts(F, MP_I32, 100, 1000, 64, MP_F32, F, 1 << 30, &o,
                                                nullptr, &h),
           MP_ERR_SIZE);
    mp_spmm_plan_free(nullptr);

    // aggregation
    expect("spmm reduce", mp_spmm(nullptr, F, MP_I32, fk<int32_t>(), nullptr, F, MP_F32, 10, 10,
                                  8, 8, 3, F, MP_F32, nullptr, MP_F32, nullptr, nullptr, 0, nullptr),
           MP_ERR_REDUCE);
    expect("spmm ldx", mp_spmm(nullptr, F, MP_I32, fk<int32_t>(), nullptr, F, MP_F32, 10, 10, 8,
                               7, MP_SUM, F, MP_F32, nullptr, MP_F32, nullptr, nullptr, 0, nullptr),
           MP_ERR_SIZE);
    expect("spmm bf16 max of f32", mp_spmm(nullptr, F, MP_I32, fk<int32_t>(), nullptr, F, MP_F32,
                                           10, 10, 8, 8, MP_MAX, nullptr, MP_F32, F, MP_BF16,
                                           fk<int32_t>(), nullptr, 0, nullptr),
           MP_ERR_DTYPE);
    expect("noalloc null col", mp_spmm_noalloc(nullptr, F, MP_I32, nullptr, nullptr, F, MP_F32,
                                               10, 10, 8, 8, MP_SUM, F, MP_F32, nullptr, MP_F32,
                                               nullptr, nullptr),
           MP_ERR_NULL);
    expect("noalloc align", mp_spmm_noalloc(nullptr, F, MP_I32, fk<int32_t>(), nullptr, fk<char>(2),
                                            MP_F32, 10, 10, 8, 8, MP_SUM, F, MP_F32, nullptr,
                                            MP_F32, nullptr, nullptr),
           MP_ERR_ALIGN);
    mp_aggr_out outs[2] = {{MP_MAX, fk<float>(), nullptr}, {MP_VAR, fk<float>(), nullptr}};
    expect("multi arg", mp_spmm_multi(nullptr, F, MP_I32, fk<int32_t>(), nullptr, F, MP_F32, 10,
                                      10, 8, 8, 2, outs, nullptr, 0, nullptr),
           MP_ERR_NULL);
    mp_aggr_out dup[2] = {{MP_VAR, fk<float>(), nullptr}, {MP_VAR, fk<float>(), nullptr}};
    expect("multi dup", mp_readout_multi(nullptr, F, MP_I32, F, MP_F32, 10, 3, 8, 8, 2, dup,
                                         nullptr, 0, nullptr),
           MP_ERR_REDUCE);
    expect("copy rows", mp_copy_rows(F, 7, F, 8, 10, 8, MP_F32, nullptr), MP_ERR_SIZE);

    // backward
    expect("transpose ws", mp_csr_transpose(F, MP_I32, fk<int32_t>(), 10, 20, 100, F, MP_I32,
                                            fk<int32_t>(), fk<int32_t>(), nullptr, nullptr, F, 16,
                                            nullptr, nullptr),
           MP_ERR_WORKSPACE);
    expect("bwx ws", mp_spmm_backward_x(nullptr, F, MP_I32, fk<int32_t>(), fk<int32_t>(), nullptr,
                                        F, MP_I32, fk<int32_t>(), F, MP_F32, 10, 10, 100, 8,
                                        MP_MAX, F, MP_F32, nullptr, 0, nullptr),
           MP_ERR_WORKSPACE);
    expect("bww reduce", mp_spmm_backward_w(F, MP_I32, fk<int32_t>(), F, MP_F32, F, MP_F32,
                                            nullptr, 10, 10, 100, 8, MP_MAX, fk<float>(), F,
                                            1 << 20, nullptr),
           MP_ERR_NULL);

    // segment matmul
    expect("gmm dims", mp_segment_matmul(seg, 3, F, F, 12, 64, F, MP_F32, F, 1 << 20, nullptr),
           MP_ERR_SIZE);
    expect("gmm bw both null", mp_segment_matmul_backward(seg, 3, F, F, F, 128, 64, nullptr,
                                                          MP_F32, nullptr, nullptr, 0, nullptr),
           MP_ERR_NULL);

    // explanation mode
    expect("csr rows", mp_csr_rows(F, MP_I32, 0, 10, fk<int32_t>(), nullptr), MP_ERR_SIZE);
    expect("msg gather dtype", mp_message_gather(fk<int32_t>(), fk<float>(), F, MP_BF16, 10, 10, 8,
                                                 F, MP_BF16, nullptr),
           MP_ERR_DTYPE);
    expect("msg scale null", mp_message_scale(nullptr, fk<float>(), 10, 8, fk<float>(), nullptr,
                                              10, nullptr),
           MP_ERR_NULL);
    expect("msg aggregate", mp_message_aggregate(nullptr, F, MP_I32, F, MP_F32, 10, 10, 8, 3, F,
                                                 MP_F32, nullptr, MP_F32, nullptr, nullptr, 0,
                                                 nullptr),
           MP_ERR_REDUCE);
    expect("msg backward", mp_message_backward(F, MP_I32, nullptr, F, MP_F32, 10, 10, 8, MP_MAX,
                                               fk<float>(), nullptr, 0, nullptr),
           MP_ERR_NULL);
    expect("edge dot", mp_edge_dot(F, MP_F32, F, MP_F32, nullptr, 10, nullptr, 10, 0, fk<float>(),
                                   nullptr),
           MP_ERR_SIZE);

    // typed graphs
    expect("hetero build null col", mp_hetero_build(2, npt, 1, &rel, 1, F, MP_I32, nullptr, F,
                                                    1 << 20, nullptr, nullptr),
           MP_ERR_NULL);
    const void* xs[2] = {F, F};
    expect("hetero reduce", mp_hetero_spmm(2, npt, xs, MP_F32, 8, 1, nullptr, F, MP_I32,
                                           fk<int32_t>(), MP_MEAN, F, MP_F32, nullptr, 0, nullptr),
           MP_ERR_REDUCE);

    // debug checks and probes
    expect("validate coo", mp_validate_coo(fk<int32_t>(), fk<int32_t>(), -1, 5, 5,
                                           fk<int64_t>(), nullptr),
           MP_ERR_SIZE);
    expect("validate csr", mp_validate_csr(F, 9, fk<int32_t>(), 5, 5, 10, fk<int64_t>(), nullptr),
           MP_ERR_DTYPE);
    expect("probe read", mp_probe_read(F, 60, fk<uint32_t>(), nullptr), MP_ERR_SIZE);
    expect("probe gather", mp_probe_gather(fk<int32_t>(), 10, F, 256, 400, fk<uint32_t>(),
                                           nullptr),
           MP_ERR_SIZE);
    if (failures) {
        std::fprintf(stderr, "%d unexpected results\n", failures);
        return 1;
    }
    std::printf("abi checks ok\n");
    return 0;
}
