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
//   pool_kernel    one workgroup per (batch, head, block): the block's Q and K
//                  rows are staged in LDS with 16-byte loads, then lane d < D
//                  sums Q column d over the rows in ascending order and lane
//                  128 + d does the same for K and divides by the token count.
//                  Writes qsum and kmean [B*H][n_blk][D].
//   select_kernel  one workgroup per (batch, head) and `rows` consecutive
//                  query blocks (8, halved until the scores fit 32 KB of
//                  LDS: 2 at 4096 blocks): the key means pass through LDS in chunks of
//                  kSelChunk blocks (one 16-byte load per lane and round), each
//                  lane scoring one (query block, key block) pair of the chunk;
//                  then one wave per row: a radix selection of the keep - 1
//                  best other blocks (independent of keep: four histogram
//                  passes over the candidates) and the kept blocks in
//                  ascending order at the row's closed-form offset (every row
//                  keeps exactly min(keep, n_blk)).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "kernels.h"

#pragma clang fp contract(off)

namespace rt {
namespace {

constexpr int kPoolThreads = 256;
constexpr int kSelThreads = 512;
constexpr int kSelRows = 8;                         // most query blocks per select workgroup
constexpr int kSelChunk = kSelThreads / kSelRows;  // key blocks per LDS chunk
constexpr int kSelScoreBytes = 32 << 10;           // LDS for the scores of one workgroup
static_assert(kSelThreads / 64 >= kSelRows, "one wave per selected row");
constexpr int kMaxD = 72;
constexpr int kPoolRows = 64;                      // largest block

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kPoolThreads) void pool_kernel(const uint16_t* __restrict__ q,
                                                            const uint16_t* __restrict__ k, int T, int D,
                                                            int block, int n_blk, float* __restrict__ qsum,
                                                            float* __restrict__ kmean) {
    // the block's rows of Q, then of K, row-major as in HBM (2D bytes per row)
    __shared__ __attribute__((aligned(16))) uint16_t tile[2][kPoolRows * kMaxD];
    const int bh = blockIdx.x / n_blk;
    const int b = blockIdx.x - bh * n_blk;
    const int t = threadIdx.x;
    const int r0 = b * block;
    const int cnt = min(block, T - r0);
    const size_t base = ((size_t)bh * T + r0) * D;
    // 16-byte pieces of the block's rows: cnt * D / 8 per tensor (D is a multiple of 8)
    const int n16 = cnt * D / 8;
    const u32x4* qs = reinterpret_cast<const u32x4*>(q + base);
    const u32x4* ks = reinterpret_cast<const u32x4*>(k + base);
    u32x4* tq = reinterpret_cast<u32x4*>(tile[0]);
    u32x4* tk = reinterpret_cast<u32x4*>(tile[1]);
    for (int i = t; i < n16; i += kPoolThreads) {
        tq[i] = qs[i];
        tk[i] = ks[i];
    }
    __syncthreads();
    const bool is_q = t < 128;
    const int d = is_q ? t : t - 128;
    if (d >= D) return;
    const uint16_t* col = tile[is_q ? 0 : 1] + d;
    float acc = 0.0f;
    for (int r = 0; r < cnt; ++r) acc = __fadd_rn(acc, bf16_to_f32(col[r * D]));
    const size_t o = ((size_t)bh * n_blk + b) * D + d;
    if (is_q) {
        qsum[o] = acc;
    } else {
        kmean[o] = __fdiv_rn(acc, (float)cnt);
    }
}

// Selection order as one unsigned key, larger = better: a NaN score counts as
// -inf and -0 as +0 (so keys are equal exactly when the fp32 scores compare
// equal), and the float's bits are mapped so that unsigned order is numeric
// order.  Equal keys go to the lower block index.
__device__ __forceinline__ uint32_t order_key(float x) {
    if (x != x) x = -INFINITY;
    if (x == 0.0f) x = 0.0f;
    const uint32_t u = __float_as_uint(x);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Number of lanes below this one whose bit is set in the wave mask m.
__device__ __forceinline__ int lanes_below(unsigned long long m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Orders the wave's LDS accesses before and after this point (one wave only:
// LDS executes a wave's instructions in issue order).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(const float* __restrict__ qsum,
                                                             const float* __restrict__ kmean, int D, int n_blk,
                                                             int keep, int rows, int32_t* __restrict__ row_ptr,
                                                             int32_t* __restrict__ col_idx) {
    // scores of the workgroup's rows: rows x n_blk floats of dynamic LDS
    extern __shared__ float sc[];
    __shared__ __attribute__((aligned(16))) float qv[kSelRows][kMaxD];  // pooled queries of the rows
    // one chunk of key means, rows padded by four floats so that the 16-byte
    // reads of 16 lanes (16 consecutive key blocks) cover the 64 banks once
    __shared__ __attribute__((aligned(16))) float km[kSelChunk * (kMaxD + 4)];
    const int n_grp = (n_blk + rows - 1) / rows;
    const int bh = blockIdx.x / n_grp;
    const int qb0 = (blockIdx.x - bh * n_grp) * rows;
    const int tid = threadIdx.x;
    const int kk = keep < n_blk ? keep : n_blk;
    const int kst = D + 4;  // LDS row stride of km (floats; a multiple of 4)
    for (int i = tid; i < rows * D; i += kSelThreads) {
        const int r = i / D, d = i - r * D;
        qv[r][d] = qb0 + r < n_blk ? qsum[((size_t)bh * n_blk + qb0 + r) * D + d] : 0.0f;
    }
    const float* kh = kmean + (size_t)bh * n_blk * D;
    const int pr = tid / kSelChunk;  // the pair this lane scores: row pr,
    const int pc = tid - pr * kSelChunk;  // key block c0 + pc
    // A chunk's nc * D floats are contiguous in HBM: 16-byte pieces i, piece
    // tid + kSelThreads j in register pf[j].  The next chunk's loads are in
    // flight while the current one is scored.
    constexpr int kPieces = (kSelChunk * kMaxD / 4 + kSelThreads - 1) / kSelThreads;
    u32x4 pf[kPieces];
    auto load_chunk = [&](int c0) {
        const int nc = n_blk - c0 < kSelChunk ? n_blk - c0 : kSelChunk;
        const int n16 = nc * D / 4;
        const u32x4* src = reinterpret_cast<const u32x4*>(kh + (size_t)c0 * D);
#pragma unroll
        for (int j = 0; j < kPieces; ++j) {
            const int i = tid + kSelThreads * j;
            if (i < n16) pf[j] = src[i];
        }
    };
    load_chunk(0);
    for (int c0 = 0; c0 < n_blk; c0 += kSelChunk) {
        const int nc = n_blk - c0 < kSelChunk ? n_blk - c0 : kSelChunk;
        __syncthreads();  // the previous chunk's scores are done (and qv is in)
        const int n16 = nc * D / 4;
#pragma unroll
        for (int j = 0; j < kPieces; ++j) {
            const int i = tid + kSelThreads * j;
            if (i < n16) {
                const int e = 4 * i, r = e / D, d = e - r * D;  // D is a multiple of 4
                *reinterpret_cast<u32x4*>(km + r * kst + d) = pf[j];
            }
        }
        __syncthreads();
        if (c0 + kSelChunk < n_blk) load_chunk(c0 + kSelChunk);
        if (pr < rows && pc < nc) {
            const u32x4* kv = reinterpret_cast<const u32x4*>(km + pc * kst);
            const u32x4* qq = reinterpret_cast<const u32x4*>(qv[pr]);
            float s = 0.0f;
            for (int d4 = 0; d4 < D / 4; ++d4) {
                const u32x4 a = qq[d4], b = kv[d4];
#pragma unroll
                for (int e = 0; e < 4; ++e) s = __fadd_rn(s, __fmul_rn(__uint_as_float(a[e]), __uint_as_float(b[e])));
            }
            sc[pr * n_blk + c0 + pc] = s;
        }
    }
    __syncthreads();
    // Selection: wave w takes row w.  Candidate block c = lane + 64 i (round
    // i).  The keep - 1 best blocks other than the diagonal are found by radix
    // selection on the 32-bit keys: four passes of 8-bit digits, from the top,
    // narrow the key of the (keep-1)-th best block (the threshold) and how many
    // blocks holding exactly that key are kept; those go to the lowest indices.
    // Every block with a larger key is kept.
    __shared__ int hist[kSelThreads / 64][256];
    const int lane = tid & 63, w = tid >> 6;
    const int qb = qb0 + w;
    if (w >= rows || qb >= n_blk) return;  // no barrier follows
    const float* row = sc + w * n_blk;
    int* hw = hist[w];
    const int n_round = (n_blk + 63) / 64;
    const int need = kk - 1;  // other blocks to keep, < n_blk
    uint32_t thr = 0, thr_mask = 0;  // digits of the threshold found so far
    int rem = need;                   // blocks still to keep at the threshold
    if (need > 0 && need < n_blk - 1) {
        for (int shift = 24; shift >= 0; shift -= 8) {
#pragma unroll
            for (int j = 0; j < 4; ++j) hw[4 * lane + j] = 0;
            wave_lds_sync();
            for (int i = 0; i < n_round; ++i) {
                const int c = lane + 64 * i;
                if (c < n_blk && c != qb) {
                    const uint32_t key = order_key(row[c]);
                    if ((key & thr_mask) == thr) atomicAdd(&hw[(key >> shift) & 255u], 1);
                }
            }
            wave_lds_sync();
            // lane L holds bins 4L .. 4L+3; S(t) counts the blocks with digit >= t
            // and the threshold's digit is the t with S(t+1) < rem <= S(t)
            int h[4], sum = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                h[j] = hw[4 * lane + j];
                sum += h[j];
            }
            int incl = sum;  // inclusive sum over lanes 0 .. lane
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int y = __shfl_up(incl, d, 64);
                if (lane >= d) incl += y;
            }
            const int tot = __shfl(incl, 63, 64);
            int s_t = tot - incl;  // bins above this lane's four
            int dig = -1, nrem = 0;
#pragma unroll
            for (int j = 3; j >= 0; --j) {
                s_t += h[j];
                if (h[j] > 0 && s_t >= rem && s_t - h[j] < rem) {
                    dig = 4 * lane + j;
                    nrem = rem - (s_t - h[j]);
                }
            }
            const unsigned long long found = __ballot(dig >= 0);
            const int src = __builtin_ctzll(found);  // exactly one lane finds it
            thr |= (uint32_t)__shfl(dig, src, 64) << shift;
            thr_mask |= 255u << shift;
            rem = __shfl(nrem, src, 64);
        }
    }
    // kept blocks in ascending order, ties at the threshold to the lowest indices
    const size_t row_off = ((size_t)bh * n_blk + qb) * kk;
    int n_tie = 0, n_out = 0;
    for (int i = 0; i < n_round; ++i) {
        const int c = lane + 64 * i;
        bool kept = false, tie = false;
        if (c < n_blk) {
            if (c == qb || need >= n_blk - 1) {
                kept = true;
            } else if (need > 0) {
                const uint32_t key = order_key(row[c]);
                tie = key == thr;
                kept = key > thr;
            }
        }
        const unsigned long long tm = __ballot(tie);
        if (tie) kept = n_tie + lanes_below(tm) < rem;
        n_tie += __popcll(tm);
        const unsigned long long km_ = __ballot(kept);
        const int pos = n_out + lanes_below(km_);
        if (kept && pos < kk) col_idx[row_off + pos] = c;  // exactly kk kept (total order)
        n_out += __popcll(km_);
    }
    if (lane == 0) {
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
    int rows = kSelRows;
    while (rows > 1 && (size_t)rows * a.n_blk * sizeof(float) > (size_t)kSelScoreBytes) rows /= 2;
    const int n_grp = (a.n_blk + rows - 1) / rows;
    const size_t lds = (size_t)rows * a.n_blk * sizeof(float);
    hipLaunchKernelGGL(select_kernel, dim3(n_bh * n_grp), dim3(kSelThreads), lds, stream, a.qsum, a.kmean, a.D,
                       a.n_blk, a.keep, rows, a.row_ptr, a.col_idx);
    return hipGetLastError();
}

}  // namespace rt
