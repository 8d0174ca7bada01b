// Streaming kernels of the statistics cache (gfx950).
//
//   cache_build    Eq.8  rho = (l_s / l_f) exp(m_s - m_f)
//                  Eq.10 R   = O_f - rho O_s
//   reshape_apply  Eq.9 with the ramp and the residual: O = min(1, rho + delta) O_s + R
//
// Without a ratio (rho == nullptr, the ablation with the reshape removed) the
// cache is R = O_f - O_s (Eq.10 with rho = 1) and the output O_s + R.
//
// Both are HBM-bound.  Each lane moves 16 bytes per tensor per step (8 bf16 of
// one row), so a wavefront reads whole 128-byte lines; rows are walked with a
// grid-stride loop over (row, 16-byte chunk) units.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace rt {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float lo_f(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Read-once / write-once 16-byte accesses, marked non-temporal so the stream
// does not displace cached data.
__device__ __forceinline__ u32x4 ld_stream(const uint16_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void st_stream(uint16_t* p, const bf16x8& v) {
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), reinterpret_cast<u32x4*>(p));
}

// Each thread takes kUnroll units a grid stride apart per trip and issues all
// their loads before any arithmetic, so kUnroll 16-byte loads per tensor are in
// flight per lane; a plain grid-stride loop finishes the remainder.
constexpr int kUnroll = 4;

template <int D>
__device__ __forceinline__ void cache_unit(int64_t row, int ch, const u32x4& f, const u32x4& s, float r,
                                           float* __restrict__ rho, uint16_t* __restrict__ resid) {
    if (ch == 0 && rho) rho[row] = r;
    bf16x8 out;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        out[2 * w] = (__bf16)(lo_f(f[w]) - r * lo_f(s[w]));
        out[2 * w + 1] = (__bf16)(hi_f(f[w]) - r * hi_f(s[w]));
    }
    st_stream(resid + (size_t)row * D + 8 * ch, out);
}

template <int D>
__global__ __launch_bounds__(256) void cache_build_kernel(const uint16_t* __restrict__ of,
                                                          const float* __restrict__ mf,
                                                          const float* __restrict__ lf,
                                                          const uint16_t* __restrict__ os,
                                                          const float* __restrict__ ms,
                                                          const float* __restrict__ ls,
                                                          int64_t rows, float* __restrict__ rho,
                                                          uint16_t* __restrict__ resid) {
    constexpr int DC = D / 8;
    const int64_t units = rows * DC;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; u + (kUnroll - 1) * stride < units; u += kUnroll * stride) {
        int64_t row[kUnroll];
        int ch[kUnroll];
        u32x4 f[kUnroll], s[kUnroll];
        float r[kUnroll];
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) {
            const int64_t uj = u + j * stride;
            row[j] = uj / DC;
            ch[j] = (int)(uj - row[j] * DC);
            const size_t off = (size_t)row[j] * D + 8 * ch[j];
            f[j] = ld_stream(of + off);
            s[j] = ld_stream(os + off);
            r[j] = rho ? (ls[row[j]] / lf[row[j]]) * expf(ms[row[j]] - mf[row[j]]) : 1.0f;
        }
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) cache_unit<D>(row[j], ch[j], f[j], s[j], r[j], rho, resid);
    }
    for (; u < units; u += stride) {
        const int64_t row = u / DC;
        const int ch = (int)(u - row * DC);
        const size_t off = (size_t)row * D + 8 * ch;
        const float r = rho ? (ls[row] / lf[row]) * expf(ms[row] - mf[row]) : 1.0f;
        cache_unit<D>(row, ch, ld_stream(of + off), ld_stream(os + off), r, rho, resid);
    }
}

template <int D>
__device__ __forceinline__ void reshape_unit(int64_t row, int ch, const u32x4& s, const u32x4& R, float r,
                                             uint16_t* __restrict__ o) {
    bf16x8 out;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        out[2 * w] = (__bf16)__builtin_fmaf(r, lo_f(s[w]), lo_f(R[w]));
        out[2 * w + 1] = (__bf16)__builtin_fmaf(r, hi_f(s[w]), hi_f(R[w]));
    }
    st_stream(o + (size_t)row * D + 8 * ch, out);
}

template <int D>
__global__ __launch_bounds__(256) void reshape_apply_kernel(const uint16_t* __restrict__ os,
                                                            const float* __restrict__ rho,
                                                            const uint16_t* __restrict__ resid,
                                                            float delta, int64_t rows,
                                                            uint16_t* __restrict__ o) {
    constexpr int DC = D / 8;
    const int64_t units = rows * DC;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; u + (kUnroll - 1) * stride < units; u += kUnroll * stride) {
        int64_t row[kUnroll];
        int ch[kUnroll];
        u32x4 s[kUnroll], R[kUnroll];
        float r[kUnroll];
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) {
            const int64_t uj = u + j * stride;
            row[j] = uj / DC;
            ch[j] = (int)(uj - row[j] * DC);
            const size_t off = (size_t)row[j] * D + 8 * ch[j];
            s[j] = ld_stream(os + off);
            R[j] = ld_stream(resid + off);
            r[j] = rho ? fminf(1.0f, rho[row[j]] + delta) : 1.0f;
        }
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) reshape_unit<D>(row[j], ch[j], s[j], R[j], r[j], o);
    }
    for (; u < units; u += stride) {
        const int64_t row = u / DC;
        const int ch = (int)(u - row * DC);
        const size_t off = (size_t)row * D + 8 * ch;
        reshape_unit<D>(row, ch, ld_stream(os + off), ld_stream(resid + off),
                        rho ? fminf(1.0f, rho[row] + delta) : 1.0f, o);
    }
}

int grid_for(int64_t units) {
    // enough workgroups to cover every CU several times; the loop strides the rest
    int64_t g = (units + 256 * kUnroll - 1) / (256 * kUnroll);
    const int64_t cap = 256 * 16;
    return (int)(g < 1 ? 1 : (g > cap ? cap : g));
}

}  // namespace

hipError_t launch_cache_build(const uint16_t* o_full, const float* m_full, const float* l_full,
                              const uint16_t* o_sparse, const float* m_sparse,
                              const float* l_sparse, int64_t rows, int D, float* rho,
                              uint16_t* resid, hipStream_t stream) {
    const int grid = grid_for(rows * (D / 8));
    if (D == 64)
        hipLaunchKernelGGL(cache_build_kernel<64>, dim3(grid), dim3(256), 0, stream, o_full, m_full,
                           l_full, o_sparse, m_sparse, l_sparse, rows, rho, resid);
    else
        hipLaunchKernelGGL(cache_build_kernel<72>, dim3(grid), dim3(256), 0, stream, o_full, m_full,
                           l_full, o_sparse, m_sparse, l_sparse, rows, rho, resid);
    return hipGetLastError();
}

hipError_t launch_reshape_apply(const uint16_t* o_sparse, const float* rho, const uint16_t* resid,
                                float rho_delta, int64_t rows, int D, uint16_t* o,
                                hipStream_t stream) {
    const int grid = grid_for(rows * (D / 8));
    if (D == 64)
        hipLaunchKernelGGL(reshape_apply_kernel<64>, dim3(grid), dim3(256), 0, stream, o_sparse, rho,
                           resid, rho_delta, rows, o);
    else
        hipLaunchKernelGGL(reshape_apply_kernel<72>, dim3(grid), dim3(256), 0, stream, o_sparse, rho,
                           resid, rho_delta, rows, o);
    return hipGetLastError();
}

}  // namespace rt
