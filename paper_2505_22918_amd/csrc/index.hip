// Block-index builder (gfx950): the static mask M of Sec.3 as a block CSR.
//
// Three launches on the caller's stream (an EXPLICIT input may stack several
// masks, one per head or per (batch, head); mask m owns row_ptr[m][0 .. n_blk]):
//   1. row_count   one workgroup per (mask, query block) writes its kept-block
//                  count into row_ptr[m][qb + 1] (closed form for the window
//                  patterns, a count of the 0/1 row for EXPLICIT);
//   2. row_scan    one workgroup turns all counts into absolute offsets in place;
//   3. row_fill    one workgroup per (mask, query block) ranks the candidate key
//                  blocks and writes the kept ones in ascending order.
//
// Ranking is exact integer arithmetic: a block's centroid is the sum of its
// token coordinates scaled by lcm / count (lcm over the candidate blocks' token
// counts), so squared distances compare exactly, and the key
// (distance^2, |kb - qb|, kb) is a total order.  Each candidate's rank is the
// number of candidates with a smaller key; a block is kept when its rank is
// below the keep count.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace rt {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxBlocks = 4096;
constexpr int kMaxRows = 32768;  // (mask, query block) rows one scan handles

__device__ int row_count_of(const IndexArgs& a, int qb) {
    if (a.kind == 1) return a.keep < a.n_blk ? a.keep : a.n_blk;
    if (a.kind == 2) {
        if (qb < a.n_tblk) return a.n_tblk;
        const int nv = a.n_blk - a.n_tblk;
        return a.n_tblk + (a.keep < nv ? a.keep : nv);
    }
    return -1;  // explicit: counted by the caller
}

__global__ __launch_bounds__(kThreads) void row_count(IndexArgs a) {
    const int m = blockIdx.x / a.n_blk;
    const int qb = blockIdx.x - m * a.n_blk;
    int32_t* const rp = a.row_ptr + (size_t)m * (a.n_blk + 1);
    __shared__ int total;
    if (a.kind != 0) {
        if (threadIdx.x == 0) rp[qb + 1] = row_count_of(a, qb);
        return;
    }
    if (threadIdx.x == 0) total = 0;
    __syncthreads();
    int n = 0;
    const uint8_t* row = a.mask + ((size_t)m * a.n_blk + qb) * a.n_blk;
    for (int kb = threadIdx.x; kb < a.n_blk; kb += kThreads) n += row[kb] != 0;
    atomicAdd(&total, n);
    __syncthreads();
    if (threadIdx.x == 0) rp[qb + 1] = total;
}

// Exclusive scan of the n_masks * n_blk row counts, in row order, into absolute
// offsets: row_ptr[m][qb] = entries of all earlier rows, row_ptr[m][n_blk] =
// row_ptr[m + 1][0] (the total after the last mask).
__global__ __launch_bounds__(kThreads) void row_scan(IndexArgs a) {
    __shared__ int cnt[kMaxRows];
    __shared__ int part[kThreads + 1];
    const int nb = a.n_blk;
    const int n = a.n_masks * nb;
    const int tid = threadIdx.x;
    for (int i = tid; i < n; i += kThreads) {
        const int m = i / nb, qb = i - m * nb;
        cnt[i] = a.row_ptr[(size_t)m * (nb + 1) + qb + 1];
    }
    __syncthreads();
    // each thread owns a contiguous segment; segment sums are scanned serially
    const int seg = (n + kThreads - 1) / kThreads;
    const int s0 = tid * seg < n ? tid * seg : n;
    const int s1 = s0 + seg < n ? s0 + seg : n;
    int local = 0;
    for (int i = s0; i < s1; ++i) local += cnt[i];
    part[tid + 1] = local;
    __syncthreads();
    if (tid == 0) {
        part[0] = 0;
        for (int i = 1; i <= kThreads; ++i) part[i] += part[i - 1];
    }
    __syncthreads();
    int run = part[tid];
    for (int i = s0; i < s1; ++i) {
        const int c = cnt[i];
        cnt[i] = run;
        run += c;
    }
    __syncthreads();
    const int total = part[kThreads];
    for (int i = tid; i < n; i += kThreads) {
        const int m = i / nb, qb = i - m * nb;
        a.row_ptr[(size_t)m * (nb + 1) + qb] = cnt[i];
    }
    for (int m = tid; m < a.n_masks; m += kThreads)
        a.row_ptr[(size_t)m * (nb + 1) + nb] = m + 1 < a.n_masks ? cnt[(m + 1) * nb] : total;
}

// scaled centroid coordinates of block b (video: b holds video tokens only)
__device__ void centroid(const IndexArgs& a, int b, int64_t c[3]) {
    const int t0 = b * a.block;
    const int t1 = (t0 + a.block < a.T) ? t0 + a.block : a.T;
    int64_t s0 = 0, s1 = 0, s2 = 0;
    if (a.kind == 1) {
        for (int t = t0; t < t1; ++t) {
            s0 += t / a.grid_w;
            s1 += t % a.grid_w;
        }
    } else {
        const int hw = a.grid_h * a.grid_w;
        for (int t = t0; t < t1; ++t) {
            const int v = t - a.n_text;
            s0 += v / hw;
            s1 += (v / a.grid_w) % a.grid_h;
            s2 += v % a.grid_w;
        }
    }
    const int64_t f = a.lcm / (t1 - t0);
    c[0] = s0 * f;
    c[1] = s1 * f;
    c[2] = s2 * f;
}

__global__ __launch_bounds__(kThreads) void row_fill(IndexArgs a) {
    __shared__ int64_t dist[kMaxBlocks];
    __shared__ uint8_t kept[kMaxBlocks];
    __shared__ int part[kThreads + 1];

    const int nb = a.n_blk;
    const int m = blockIdx.x / nb;
    const int qb = blockIdx.x - m * nb;
    const int tid = threadIdx.x;

    // candidate range and how many of them to keep
    int lo = 0, k = 0;
    bool ranked = false;
    if (a.kind == 1) {
        ranked = true;
        k = a.keep < nb ? a.keep : nb;
    } else if (a.kind == 2 && qb >= a.n_tblk) {
        ranked = true;
        lo = a.n_tblk;
        k = a.keep < nb - lo ? a.keep : nb - lo;
    }

    if (ranked) {
        int64_t cq[3];
        centroid(a, qb, cq);
        for (int kb = lo + tid; kb < nb; kb += kThreads) {
            int64_t ck[3];
            centroid(a, kb, ck);
            const int64_t d0 = ck[0] - cq[0], d1 = ck[1] - cq[1], d2 = ck[2] - cq[2];
            dist[kb] = d0 * d0 + d1 * d1 + d2 * d2;
        }
        __syncthreads();
        for (int kb = lo + tid; kb < nb; kb += kThreads) {
            const int64_t dk = dist[kb];
            const int ak = kb > qb ? kb - qb : qb - kb;
            int rank = 0;
            for (int j = lo; j < nb; ++j) {
                const int64_t dj = dist[j];
                const int aj = j > qb ? j - qb : qb - j;
                rank += (dj < dk) || (dj == dk && (aj < ak || (aj == ak && j < kb)));
            }
            kept[kb] = rank < k;
        }
        // text key blocks of a video row are always kept
        for (int kb = tid; kb < lo; kb += kThreads) kept[kb] = 1;
    } else if (a.kind == 2) {
        // text query block: text key blocks only
        for (int kb = tid; kb < nb; kb += kThreads) kept[kb] = kb < a.n_tblk;
    } else {
        const uint8_t* row = a.mask + ((size_t)m * nb + qb) * nb;
        for (int kb = tid; kb < nb; kb += kThreads) kept[kb] = row[kb] != 0;
    }
    __syncthreads();

    // ordered write: each thread owns a contiguous segment of key blocks
    const int seg = (nb + kThreads - 1) / kThreads;
    const int s0 = tid * seg;
    const int s1 = (s0 + seg < nb) ? s0 + seg : nb;
    int n = 0;
    for (int kb = s0; kb < s1; ++kb) n += kept[kb];
    part[tid + 1] = n;
    __syncthreads();
    if (tid == 0) {
        part[0] = 0;
        for (int i = 1; i <= kThreads; ++i) part[i] += part[i - 1];
    }
    __syncthreads();
    int pos = a.row_ptr[(size_t)m * (nb + 1) + qb] + part[tid];
    for (int kb = s0; kb < s1; ++kb) {
        if (kept[kb]) {
            if (pos >= 0 && pos < a.capacity) a.col_idx[pos] = kb;
            ++pos;
        }
    }
}

}  // namespace

hipError_t launch_index_build(const IndexArgs& a, hipStream_t stream) {
    const int rows = a.n_masks * a.n_blk;
    hipLaunchKernelGGL(row_count, dim3(rows), dim3(kThreads), 0, stream, a);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(row_scan, dim3(1), dim3(kThreads), 0, stream, a);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(row_fill, dim3(rows), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace rt
