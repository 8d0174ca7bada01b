// Dynamic block mask (gfx950): the kept key blocks chosen at run time from the
// step's own Q and K, one mask per (batch, head), in the stacked CSR layout the
// attention kernels take (n_masks = B*H).
//
// The paper keeps a static mask and names run-time masks as future work,
// adapted to attention statistics or token importance (Sec.6, App. A.2); the
// dynamic methods it cites pool Q K^T into blocks and keep the top-scoring
// blocks (Sec.2).  The rule built here, per (batch, head) and query block qb:
//   score(qb, kb) = sum_d Qsum_qb[d] * Kmean_kb[d]
// with Qsum the fp32 sum of qb's rows (one addition per row, ascending), Kmean
// the fp32 sum of kb's rows (same order) divided by its token count, and the
// dot product accumulated in fp32 over ascending d with the product and the sum
// rounded separately.  qb keeps itself (Eq.5 needs a non-empty kept set) and
// the keep - 1 best other blocks (higher score first, ties to the lower index,
// a NaN score ranked last); rows are stored ascending.  Every fp32 operation is
// fixed, so the choice is reproducible bit for bit.
//
//   pool_kernel    one workgroup per (batch, head, block): lane d < D sums the
//                  block's Q rows, lane 128 + d its K rows; the K sum is divided
//                  by the token count.  Writes qsum and kmean [B*H][n_blk][D].
//   select_kernel  one workgroup per (batch, head, query block): every key
//                  block's score into LDS, each candidate's rank among the other
//                  blocks, then the kept blocks in ascending order at the row's
//                  closed-form offset (every row keeps exactly min(keep, n_blk)).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "kernels.h"

#pragma clang fp contract(off)

namespace rt {
namespace {

constexpr int kPoolThreads = 256;
constexpr int kSelThreads = 256;
constexpr int kMaxDynBlocks = 4096;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__global__ __launch_bounds__(kPoolThreads) void pool_kernel(const uint16_t* __restrict__ q,
                                                            const uint16_t* __restrict__ k, int T, int D,
                                                            int block, int n_blk, float* __restrict__ qsum,
                                                            float* __restrict__ kmean) {
    const int bh = blockIdx.x / n_blk;
    const int b = blockIdx.x - bh * n_blk;
    const int t = threadIdx.x;
    const bool is_q = t < 128;
    const int d = is_q ? t : t - 128;
    if (d >= D) return;
    const int r0 = b * block;
    const int cnt = min(block, T - r0);
    const uint16_t* src = (is_q ? q : k) + ((size_t)bh * T + r0) * D + d;
    float acc = 0.0f;
    for (int r = 0; r < cnt; ++r) acc = __fadd_rn(acc, bf16_to_f32(src[(size_t)r * D]));
    const size_t o = ((size_t)bh * n_blk + b) * D + d;
    if (is_q) {
        qsum[o] = acc;
    } else {
        kmean[o] = __fdiv_rn(acc, (float)cnt);
    }
}

// a > b in the selection order: higher score first, a NaN score last, then the
// lower block index
__device__ __forceinline__ bool before(float sa, int a, float sb, int b) {
    const float xa = sa != sa ? -INFINITY : sa;
    const float xb = sb != sb ? -INFINITY : sb;
    return xa > xb || (xa == xb && a < b);
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(const float* __restrict__ qsum,
                                                             const float* __restrict__ kmean, int D, int n_blk,
                                                             int keep, int32_t* __restrict__ row_ptr,
                                                             int32_t* __restrict__ col_idx) {
    __shared__ float sc[kMaxDynBlocks];
    __shared__ float qv[128];
    __shared__ int part[kSelThreads + 1];
    const int bh = blockIdx.x / n_blk;
    const int qb = blockIdx.x - bh * n_blk;
    const int tid = threadIdx.x;
    const int kk = keep < n_blk ? keep : n_blk;
    if (tid < D) qv[tid] = qsum[((size_t)bh * n_blk + qb) * D + tid];
    __syncthreads();
    for (int kb = tid; kb < n_blk; kb += kSelThreads) {
        const float* km = kmean + ((size_t)bh * n_blk + kb) * D;
        float s = 0.0f;
        for (int d = 0; d < D; ++d) s = __fadd_rn(s, __fmul_rn(qv[d], km[d]));
        sc[kb] = s;
    }
    __syncthreads();
    // each thread owns a contiguous run of candidate blocks; a block is kept when
    // it is the diagonal or ranks among the keep - 1 best other blocks
    const int seg = (n_blk + kSelThreads - 1) / kSelThreads;
    const int c0 = tid * seg < n_blk ? tid * seg : n_blk;
    const int c1 = c0 + seg < n_blk ? c0 + seg : n_blk;
    unsigned long long kept_bits = 0;  // bit i: candidate c0 + i is kept (seg <= 16)
    int n_kept = 0;
    for (int c = c0; c < c1; ++c) {
        bool kept = c == qb;
        if (!kept && kk > 1) {
            int rank = 0;
            const float s = sc[c];
            for (int o = 0; o < n_blk && rank < kk - 1; ++o) rank += (o != qb && o != c && before(sc[o], o, s, c));
            kept = rank < kk - 1;
        }
        if (kept) {
            kept_bits |= 1ull << (c - c0);
            ++n_kept;
        }
    }
    part[tid + 1] = n_kept;
    if (tid == 0) part[0] = 0;
    __syncthreads();
    if (tid == 0) {
        for (int i = 1; i <= kSelThreads; ++i) part[i] += part[i - 1];
    }
    __syncthreads();
    const size_t row_off = ((size_t)bh * n_blk + qb) * kk;
    int pos = part[tid];
    for (int c = c0; c < c1; ++c) {
        if ((kept_bits >> (c - c0)) & 1ull) {
            if (pos < kk) col_idx[row_off + pos] = c;  // exactly kk kept per row (total order)
            ++pos;
        }
    }
    if (tid == 0) {
        row_ptr[(size_t)bh * (n_blk + 1) + qb] = (int32_t)row_off;
        if (qb == n_blk - 1) row_ptr[(size_t)bh * (n_blk + 1) + n_blk] = (int32_t)(row_off + kk);
    }
}

constexpr int kMaxDevices = 64;
std::atomic<float*> g_scratch_ptr[kMaxDevices];

}  // namespace

// Library-owned workspace of rt_dynamic_index_noalloc, for callers that cannot
// allocate: the pooled query sums and key means, 2 * B*H*n_blk*D floats at most
// kDynScratchFloats (16 MiB).  Each GPU holds its own copy until the process
// ends.  In host code `scratch` names a host-side stand-in, never the device
// memory: its device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) float scratch[kDynScratchFloats];

hipError_t dynamic_scratch(float** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    float* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        // first call on this device, with it current: its copy's address
        void* addr = nullptr;
        e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        p = static_cast<float*>(addr);
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *ptr = p;
    return hipSuccess;
}

hipError_t launch_dynamic_index(const DynIndexArgs& a, hipStream_t stream) {
    const int n_bh = a.B * a.H;
    hipLaunchKernelGGL(pool_kernel, dim3(n_bh * a.n_blk), dim3(kPoolThreads), 0, stream, a.q, a.k, a.T, a.D,
                       a.block, a.n_blk, a.qsum, a.kmean);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(select_kernel, dim3(n_bh * a.n_blk), dim3(kSelThreads), 0, stream, a.qsum, a.kmean, a.D,
                       a.n_blk, a.keep, a.row_ptr, a.col_idx);
    return hipGetLastError();
}

}  // namespace rt
