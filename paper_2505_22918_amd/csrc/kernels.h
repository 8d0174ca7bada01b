// Internal launch interface between the C ABI (api.cpp) and the HIP kernels.
// Arguments reaching these launchers have already been validated on the host.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rt {

struct AttnArgs {
    const uint16_t* q;  // bf16 [B,H,T,D]
    const uint16_t* k;
    const uint16_t* v;
    uint16_t* o;        // bf16 [B,H,T,D]
    float* row_max;     // fp32 [B,H,T] or null
    float* row_sum;     // fp32 [B,H,T] or null
    const float* rho;   // reshape only: fp32 [B,H,T]
    const uint16_t* resid;  // reshape only: bf16 [B,H,T,D]
    float rho_delta;
    const int32_t* row_ptr;  // sparse only: [n_masks][n_blk + 1], absolute offsets
    const int32_t* col_idx;
    int32_t nnz;
    int32_t n_masks;    // 1: shared; H: per head; B*H: per (batch, head)
    int32_t heads;      // H
    int32_t T;
    int32_t n_blk;      // ceil(T / block)
    int32_t dense;      // 1: walk every key block, ignore the CSR
    int32_t n_items;    // B*H*n_blk workgroups of real work
    int32_t per_xcd;    // ceil(n_items / 8)
    float scale_log2;   // log2(e) / sqrt(D)
    float scale_nat;    // 1 / sqrt(D)
    float* rho_out;     // caching step only: fp32 [B,H,T]
    uint16_t* resid_out;  // caching step only: bf16 [B,H,T,D]
    int32_t postmask;   // caching walk only: write (A o M) V (Eq.7) to o instead of O_full, rho, R
};

// What one launch computes: attention over the kept blocks (or every block when
// dense), the same with the reshape epilogue, or the one-pass caching step
// (every block, with the kept / not-kept split of the CSR).
enum AttnMode { kAttn = 0, kAttnReshape = 1, kAttnCache = 2 };

hipError_t launch_attention(const AttnArgs& a, int D, int block, AttnMode mode, hipStream_t stream);

hipError_t launch_cache_build(const uint16_t* o_full, const float* m_full, const float* l_full,
                              const uint16_t* o_sparse, const float* m_sparse,
                              const float* l_sparse, int64_t rows, int D, float* rho,
                              uint16_t* resid, hipStream_t stream);

hipError_t launch_reshape_apply(const uint16_t* o_sparse, const float* rho, const uint16_t* resid,
                                float rho_delta, int64_t rows, int D, uint16_t* o,
                                hipStream_t stream);

struct IndexArgs {
    int32_t kind;
    const uint8_t* mask;  // EXPLICIT, device
    int32_t T, block, n_blk;
    int32_t grid_h, grid_w, frames, n_text;
    int32_t keep;
    int32_t n_masks;      // EXPLICIT masks stacked in `mask`
    int32_t n_tblk;       // VIDEO3D text blocks
    int64_t lcm;          // lcm of candidate block token counts
    int32_t* row_ptr;
    int32_t* col_idx;
    int32_t capacity;
};

hipError_t launch_index_build(const IndexArgs& a, hipStream_t stream);

// Dynamic block mask from the step's Q and K (dynamic.hip): workspace qsum and
// kmean [B*H][n_blk][D] fp32; row_ptr [B*H][n_blk + 1], col_idx [B*H*n_blk*kk]
// with kk = min(keep, n_blk).
struct DynIndexArgs {
    const uint16_t* q;  // bf16 [B,H,T,D]
    const uint16_t* k;
    int32_t B, H, T, D;
    int32_t block, n_blk, keep;
    float* qsum;
    float* kmean;
    int32_t* row_ptr;
    int32_t* col_idx;
};

hipError_t launch_dynamic_index(const DynIndexArgs& a, hipStream_t stream);

// The library-owned workspace of the allocation-free dynamic index build: the
// device address of this GPU's copy (looked up on the first call on a device).
constexpr int64_t kDynScratchFloats = (int64_t)4 << 20;  // 16 MiB
hipError_t dynamic_scratch(float** ptr);

}  // namespace rt
