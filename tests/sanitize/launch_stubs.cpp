// Host-only stand-ins for the kernel launchers of csrc/kernels.h, so that the C
// ABI (csrc/api.cpp) can be built with the host compiler under AddressSanitizer
// and UndefinedBehaviorSanitizer and driven by the ABI tests without a GPU.
// Each stand-in checks what the validation layer hands it and launches nothing;
// a violated expectation aborts the process.
#include <hip/hip_runtime_api.h>

#include <cstdio>
#include <cstdlib>

#include "kernels.h"

#define EXPECT(c)                                                                  \
    do {                                                                           \
        if (!(c)) {                                                                \
            std::fprintf(stderr, "launch stub: expectation failed: %s\n", #c);    \
            std::abort();                                                          \
        }                                                                          \
    } while (0)

extern "C" const char* hipGetErrorString(hipError_t) { return "hip (stubbed)"; }

namespace rt {

hipError_t launch_attention(const AttnArgs& a, int D, int block, AttnMode mode, hipStream_t) {
    EXPECT(D == 64 || D == 72);
    EXPECT(block == 32 || block == 64);
    EXPECT(a.q && a.k && a.v && a.o);
    EXPECT(a.T > 0 && a.n_blk == (a.T + block - 1) / block);
    EXPECT(a.n_items > 0 && a.n_items % a.n_blk == 0);
    EXPECT(8LL * a.per_xcd >= a.n_items && 8LL * (a.per_xcd - 1) < a.n_items);
    EXPECT((long long)a.T * D * 2 <= (1LL << 30));
    if (!a.dense) {
        EXPECT(a.row_ptr && a.col_idx && a.nnz > 0 && a.n_masks >= 1);
    }
    if (mode == kAttnReshape) EXPECT(a.resid);  // rho may be absent (no ratio)
    if (mode == kAttnCache && !a.postmask) EXPECT(a.resid_out);
    return hipSuccess;
}

hipError_t launch_cache_build(const uint16_t* o_full, const float* m_full, const float* l_full,
                              const uint16_t* o_sparse, const float* m_sparse, const float* l_sparse,
                              int64_t rows, int D, float* rho, uint16_t* resid, hipStream_t) {
    EXPECT(o_full && o_sparse && resid);
    if (rho) EXPECT(m_full && l_full && m_sparse && l_sparse);
    EXPECT(rows > 0 && (D == 64 || D == 72));
    return hipSuccess;
}

hipError_t launch_reshape_apply(const uint16_t* o_sparse, const float* rho, const uint16_t* resid,
                                float, int64_t rows, int D, uint16_t* o, hipStream_t) {
    EXPECT(o_sparse && resid && o && rows > 0 && (D == 64 || D == 72));
    return hipSuccess;
}

hipError_t launch_index_build(const IndexArgs& a, hipStream_t) {
    EXPECT(a.row_ptr && a.col_idx && a.T > 0 && a.n_blk == (a.T + a.block - 1) / a.block);
    EXPECT(a.n_blk <= 4096 && a.n_masks >= 1 && a.capacity >= 0);
    if (a.kind == 0) EXPECT(a.mask);
    return hipSuccess;
}

hipError_t launch_dynamic_index(const DynIndexArgs& a, hipStream_t) {
    EXPECT(a.q && a.k && a.qsum && a.kmean && a.row_ptr && a.col_idx);
    EXPECT(a.T > 0 && a.n_blk == (a.T + a.block - 1) / a.block && a.n_blk <= 4096 && a.keep >= 1);
    EXPECT(a.kmean == a.qsum + (size_t)a.B * a.H * a.n_blk * a.D);
    return hipSuccess;
}

hipError_t dynamic_scratch(float** ptr) {
    static float stand_in[4];  // the sanitizer build never launches, so no device memory is needed
    *ptr = stand_in;
    return hipSuccess;
}

}  // namespace rt
