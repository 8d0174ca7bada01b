// Block-sparse / dense softmax attention with row statistics and the fused
// Re-ttention reshape epilogue, for gfx950 (CDNA4).
//
//   rt_attn_full            Eq.1 with the Eq.4 denominator, every key block
//   rt_attn_sparse          Eq.5, the kept key blocks of a block CSR
//   rt_attn_sparse_reshape  Eq.5, then Eq.9 (rho, ramped) and Eq.10 (residual)
//
// One workgroup is one wavefront that owns one query block (32 or 64 rows) of
// one (batch, head) and walks the key blocks of its CSR row in 32-key chunks:
//
//   S^T = K_chunk Q^T          v_mfma_f32_32x32x16_bf16, keys x queries
//   online softmax             fp32, exp2 with log2(e)/sqrt(D) folded in
//   O^T += V_chunk^T P^T       v_mfma_f32_32x32x16_bf16, head-dim x queries
//
// Computing the transposed products keeps every query in one lane column: the
// 32x32 accumulator of S^T hands each lane 16 keys of one query, which are
// exactly the 8+8 key values the B operand of the P V product needs, so P
// never leaves registers.  The row max needs one exchange between lane l and
// l^32 (v_permlane32_swap).
//
// Memory.  K and V chunks move from HBM/L2 straight into a two-stage LDS ring
// with buffer_load ... lds (no staging registers); chunk i+1 is in flight while
// chunk i is computed.  A buffer resource per chunk ends at the last key row,
// so rows past T arrive as zeros (their scores are then masked to -inf).  Rows
// stay row-major in LDS: K is read as the A operand with 16-byte reads, V^T
// through ds_read_b64_tr_b16, the CDNA4 LDS transpose read.  16-byte slots of a
// row are XOR-swizzled by row so both reads are free of bank conflicts (72-wide
// heads use 144-byte rows, which spread banks as is).  The first chunk's DMA is
// in flight together with the Q and rho loads; once the last chunk has been
// issued, the residual tile R of the query block is brought into the stage that
// falls free, so the epilogue finds it in LDS.
//
// Softmax.  The running max m_run starts at the first chunk's max and moves
// only when a chunk's probabilities against it reach 2^64 (far below fp32 and
// bf16 overflow); that rare case rescales O and l and recomputes the chunk.
// Without requested statistics no per-chunk max is taken at all: the overflow
// test reads the chunk's row sum.  With statistics the exact max is tracked and
// l is moved to it at the end, so the emitted pair is exactly max and exp-sum.
//
// Epilogue.  O = factor * acc (+ R) is formed in registers against R read from
// LDS, written back as bf16 over R in place, and leaves as 16-byte row stores.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace rt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) int32_t* csr_ptr;
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

constexpr float kJump = 18446744073709551616.0f;  // 2^64: stale-max limit on a probability

// Geometry of one 32-key chunk of K or V in LDS.
template <int D>
struct Geo;
template <>
struct Geo<64> {
    static constexpr int DK = 64;      // Q K^T contraction width (multiple of 16)
    static constexpr int DV = 64;      // rows of O^T (multiple of 32)
    static constexpr int SLOTS = 8;    // 16-byte slots per row
    static constexpr bool SWZ = true;  // XOR-swizzle slots by row
};
template <>
struct Geo<72> {
    static constexpr int DK = 80;
    static constexpr int DV = 96;
    static constexpr int SLOTS = 9;
    static constexpr bool SWZ = false;
};

// K rows (and the R / O tile): 8 consecutive rows read the same slot -> XOR with r & 7.
template <int D>
__device__ __forceinline__ int kswz(int r) {
    return Geo<D>::SWZ ? (r & 7) : 0;
}
// V rows: a transpose read covers 4 consecutive rows x 2 adjacent slots -> XOR
// with 2 * (r & 3) keeps those 8 (row, slot) pairs on distinct banks.
template <int D>
__device__ __forceinline__ int vswz(int r) {
    return Geo<D>::SWZ ? ((r & 3) << 1) : 0;
}

__device__ __forceinline__ float pair_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float lo_f(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
    const bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)0.f, (__bf16)0.f};
    return __builtin_bit_cast(u32x2, v)[0];
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14]).
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// 16 bytes per lane from buffer `rsrc` at byte offset `voff` into LDS at
// m0 + 16 * lane (buffer_load_dwordx4 ... lds).  m0 is reserved by the compiler
// (never allocated) and is set before every use.  Issued from inline assembly so
// the compiler neither orders these loads against LDS reads of other stages nor
// waits for them; the kernel waits on the vector-memory counter itself.
__device__ __forceinline__ void dma16(uint32_t lds_addr, int voff, i32x4 rsrc) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(rsrc)
        : "memory");
}

__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, int bytes) {
    const uint64_t p = (uint64_t)(uintptr_t)base;
    return i32x4{(int)(uint32_t)p, (int)((uint32_t)(p >> 32) & 0xffffu), bytes, 0x00020000};
}

template <int D, int BS>
constexpr int kWaves = (D == 72 && BS == 64) ? 1 : 2;

template <int D, int BS, bool RESHAPE, bool STATS>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(kWaves<D, BS>)))
void attn_fwd(AttnArgs a) {
    using G = Geo<D>;
    constexpr int DK = G::DK;
    constexpr int DV = G::DV;
    constexpr int QT = BS / 32;              // 32-query tiles per workgroup
    constexpr int DS = DK / 16;              // k-steps of Q K^T
    constexpr int DT = DV / 32;              // 32-row tiles of O^T
    constexpr int DC = D / 8;                // 16-byte chunks per token row
    constexpr int ROWB = G::SLOTS * 16;      // LDS bytes per K / V / R row (= 2 * D)
    constexpr int TILE = 32 * ROWB;          // LDS bytes per K or V chunk
    constexpr int STAGE = 2 * TILE;          // one ring stage: K then V
    constexpr int NSLOT = 32 * G::SLOTS;     // 16-byte slots per chunk and tensor
    constexpr int NDMA = (NSLOT + 63) / 64;  // DMA instructions per chunk and tensor
    constexpr int RSLOT = BS * DC;           // 16-byte slots of the R tile
    constexpr int NDMA_R = (RSLOT + 63) / 64;
    constexpr int SMEM = 2 * STAGE + 256;    // two stages + slack for padded V^T reads
    static_assert(RSLOT * 16 <= STAGE, "R tile fits a stage");
    static_assert(ROWB == 2 * D, "rows are unpadded");

    __shared__ __attribute__((aligned(1024))) unsigned char smem[SMEM];
    lds_u8* const lds = (lds_u8*)smem;
    const uint32_t lds0 = (uint32_t)(uintptr_t)lds;

    const int lane = threadIdx.x;
    const int l32 = lane & 31;
    const int hi = lane >> 5;

    // XCD-aware order: hardware workgroup g runs on XCD g % 8; give each XCD a
    // contiguous run of (head, query block) items so a head's K/V stays in one L2.
    const int g = blockIdx.x;
    const int item = (g & 7) * a.per_xcd + (g >> 3);
    if (item >= a.n_items) return;
    const int bh = item / a.n_blk;
    const int qb = item - bh * a.n_blk;
    const int T = a.T;
    const size_t head_off = (size_t)bh * (size_t)T * D;
    const uint16_t* __restrict__ Kh = a.k + head_off;
    const uint16_t* __restrict__ Vh = a.v + head_off;
    const int row0 = qb * BS;  // first query row of the block

    // ---- per-lane constant offsets ------------------------------------------------
    // DMA: lane fills 16-byte LDS slot n*64 + lane of a chunk, i.e. (row r, slot s),
    // from global (row r, head-dim chunk s ^ swizzle(r)).
    int kdma[NDMA], vdma[NDMA];
#pragma unroll
    for (int n = 0; n < NDMA; ++n) {
        const int slot = n * 64 + lane;
        const int r = slot / G::SLOTS, s = slot - (slot / G::SLOTS) * G::SLOTS;
        kdma[n] = r * (D * 2) + ((s ^ kswz<D>(r)) * 16);
        vdma[n] = r * (D * 2) + ((s ^ vswz<D>(r)) * 16);
    }
    // K A-operand reads: row l32, head-dim chunk 2s + hi (clamped to the last real
    // chunk for a 72-wide head, where the matching Q values are zero)
    int k_rd[DS];
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        int ch = 2 * s + hi;
        ch = ch < DC ? ch : DC - 1;
        k_rd[s] = l32 * ROWB + ((ch ^ kswz<D>(l32)) * 16);
    }
    // V^T A-operand transpose reads: in each group of 16 lanes, lane L supplies row
    // 4*hi + L/4 (+16ks, +8 for the second read) at head-dim 32dt + 16(group & 1) +
    // 4(L & 3); every lane then receives 4 consecutive rows at head-dim 32dt + l32.
    int v_rd[DT];
    {
        const int G4 = lane >> 4, L = lane & 15;
        const int r = 4 * hi + (L >> 2);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const int d = 32 * dt + 16 * (G4 & 1) + 4 * (L & 3);
            v_rd[dt] = r * ROWB + (((d >> 3) ^ vswz<D>(r)) * 16) + (d & 7) * 2;
        }
    }

    // ---- kept key blocks of this query block ----------------------------------------
    int e_beg, e_end;
    if (a.dense) {
        e_beg = 0;
        e_end = a.n_blk;
    } else {
        e_beg = ((csr_ptr)a.row_ptr)[qb];
        e_end = ((csr_ptr)a.row_ptr)[qb + 1];
        e_beg = e_beg < 0 ? 0 : (e_beg > a.nnz ? a.nnz : e_beg);
        e_end = e_end < e_beg ? e_beg : (e_end > a.nnz ? a.nnz : e_end);
    }
    // The walk visits chunk i = 0 .. n_chunk-1: kept entry i / (BS/32), 32-key
    // half i % (BS/32).  A chunk holding no key (an entry outside [0, n_blk), or
    // the empty half of a short last block) is not loaded and is fully masked.
    // The first 64 column indices live in one VGPR (lane j holds entry e_beg + j);
    // longer rows read the rest with scalar loads.
    int cols = -1;
    if (!a.dense && lane < e_end - e_beg) cols = ((csr_ptr)a.col_idx)[e_beg + lane];
    const int n_chunk = (e_end - e_beg) * (BS / 32);
    auto chunk_base = [&](int i) -> int {
        const int j = i / (BS / 32), half = i - j * (BS / 32);
        int kb;
        if (a.dense) {
            kb = j;
        } else if (j < 64) {
            kb = __builtin_amdgcn_readlane(cols, j);
        } else {
            kb = ((csr_ptr)a.col_idx)[e_beg + j];
        }
        const int base = kb * BS + 32 * half;
        return (kb >= 0 && kb < a.n_blk && base < T) ? base : -1;
    };

    // DMA of the 32-key K and V chunks starting at key `base` into ring stage `st`;
    // the buffers end at row T, so rows past it read as zeros.
    auto issue = [&](int base, int st) {
        if (base < 0) return;
        const int left = (T - base) * (D * 2);
        const int nrec = left < 32 * D * 2 ? left : 32 * D * 2;
        const i32x4 kr = buffer_rsrc(Kh + (size_t)base * D, nrec);
        const i32x4 vr = buffer_rsrc(Vh + (size_t)base * D, nrec);
#pragma unroll
        for (int n = 0; n < NDMA; ++n) {
            if (NSLOT % 64 == 0 || n * 64 + lane < NSLOT) dma16(lds0 + st * STAGE + n * 1024, kdma[n], kr);
        }
#pragma unroll
        for (int n = 0; n < NDMA; ++n) {
            if (NSLOT % 64 == 0 || n * 64 + lane < NSLOT)
                dma16(lds0 + st * STAGE + TILE + n * 1024, vdma[n], vr);
        }
    };
    // DMA of the block's residual rows into ring stage `st`, same row layout and
    // swizzle as K (rows past T read as zeros)
    auto issue_r = [&](int st) {
        const int left = (T - row0) * (D * 2);
        const int nrec = left < BS * D * 2 ? left : BS * D * 2;
        const i32x4 rr = buffer_rsrc(a.resid + head_off + (size_t)row0 * D, nrec);
#pragma unroll
        for (int n = 0; n < NDMA_R; ++n) {
            const int slot = n * 64 + lane;
            const int r = slot / DC, s = slot - (slot / DC) * DC;
            if (RSLOT % 64 == 0 || slot < RSLOT)
                dma16(lds0 + st * STAGE + n * 1024, r * (D * 2) + ((s ^ kswz<D>(r)) * 16), rr);
        }
    };

    // ---- prologue: first chunk's DMA, Q, rho in flight together --------------------
    int cur = n_chunk > 0 ? chunk_base(0) : -1;
    int nxt = n_chunk > 1 ? chunk_base(1) : -1;
    issue(cur, 0);

    float rho_r[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int row = row0 + qt * 32 + l32;
        rho_r[qt] = (RESHAPE && row < T) ? a.rho[(size_t)bh * T + row] : 0.f;
    }
    // Q^T operands: lane holds query l32 of tile qt, head dims 16s + 8hi .. +7
    bf16x8 qop[QT][DS];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        int row = row0 + qt * 32 + l32;
        row = row < T ? row : T - 1;
        const uint16_t* qr = a.q + head_off + (size_t)row * D;
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            const int d0 = 16 * s + 8 * hi;
            if (d0 < D) {
                qop[qt][s] = *reinterpret_cast<const bf16x8*>(qr + d0);
            } else {
                qop[qt][s] = bf16x8{};
            }
        }
    }
    wait_vm<0>();  // chunk 0, Q, rho and the CSR window have landed
    issue(nxt, 1);

    const float c2 = a.scale_log2;  // log2(e) / sqrt(D)
    f32x16 oacc[QT][DT];
    float m_run[QT], m_top[QT], l_run[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        m_run[qt] = -1e30f;  // finite: a fully masked chunk then yields p = 0, not NaN
        m_top[qt] = -INFINITY;
        l_run[qt] = 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[qt][dt] = f32x16{};
    }

    // probabilities of one 32-key chunk against the running max: bf16 operand for
    // P V and the fp32 row sum of the lane's 16 keys
    auto probs = [&](const f32x16& sc, float mrun, bf16x8 (&pp)[2]) {
        const float mc = mrun * c2;
        float lsum = 0.f;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
            for (int x = 0; x < 8; ++x) {
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[8 * ks + x], c2, -mc));
                lsum += p;
                pp[ks][x] = (__bf16)p;
            }
        }
        return lsum;
    };
    // row max of one chunk; lane holds keys 8j + 4hi + i for acc index 4j + i, the
    // other 16 keys of its query sit in lane l ^ 32
    auto chunk_max = [&](const f32x16& sc) {
        float mx = fmaxf(fmaxf(sc[0], sc[1]), sc[2]);
#pragma unroll
        for (int x = 3; x < 15; x += 2) mx = fmaxf(fmaxf(mx, sc[x]), sc[x + 1]);
        mx = fmaxf(mx, sc[15]);
        return pair_max(mx);
    };

    int st = 0;     // ring stage of chunk cur
    int r_st = -1;  // stage the residual tile was brought into
    for (int i = 0; i < n_chunk; ++i) {
        const lds_u8* Ks = lds + st * STAGE;
        const lds_u8* Vs = Ks + TILE;

        // S^T = K Q^T
        f32x16 sacc[QT];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) sacc[qt] = f32x16{};
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            const bf16x8 kop = *(const lds_bf16x8*)(Ks + k_rd[s]);
#pragma unroll
            for (int qt = 0; qt < QT; ++qt)
                sacc[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[qt][s], sacc[qt], 0, 0, 0);
        }
        if (cur < 0 || cur + 32 > T) {  // keys past T, or a chunk holding no key
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
                for (int x = 0; x < 16; ++x) {
                    const int key = cur + 8 * (x >> 2) + 4 * hi + (x & 3);
                    if (cur < 0 || key >= T) sacc[qt][x] = -INFINITY;
                }
            }
        }

        // softmax against the stale max; the rare overflow case takes the slow path
        bf16x8 pop[QT][2];
        float lsum[QT];
        float mx[QT];
        bool jump = false;
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            if (STATS) {
                mx[qt] = chunk_max(sacc[qt]);
                m_top[qt] = fmaxf(m_top[qt], mx[qt]);
            }
            lsum[qt] = probs(sacc[qt], m_run[qt], pop[qt]);
            jump |= !(lsum[qt] < kJump);
        }
        if (__builtin_amdgcn_ballot_w64(jump)) {
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
                if (!STATS) mx[qt] = chunk_max(sacc[qt]);
                const float mnew = fmaxf(m_run[qt], mx[qt]);
                const float alpha = __builtin_amdgcn_exp2f((m_run[qt] - mnew) * c2);
                l_run[qt] *= alpha;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) oacc[qt][dt] *= alpha;
                m_run[qt] = mnew;
                lsum[qt] = probs(sacc[qt], m_run[qt], pop[qt]);
            }
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) l_run[qt] += lsum[qt];

        // O^T += V^T P^T; the V^T operand is two transpose reads of 4 rows each
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(Vs + v_rd[dt] + 16 * ks * ROWB));
                const bf16x4 v1 =
                    __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(Vs + v_rd[dt] + (16 * ks + 8) * ROWB));
                const bf16x8 vv = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
                for (int qt = 0; qt < QT; ++qt)
                    oacc[qt][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vv, pop[qt][ks], oacc[qt][dt], 0, 0, 0);
            }
        }

        // refill the stage just consumed: chunk i+2, or the residual tile once the
        // chunk sequence is exhausted; then wait for chunk i+1
        const bool more = i + 2 < n_chunk;
        const int nx2 = more ? chunk_base(i + 2) : -1;
        if (nx2 >= 0) {
            issue(nx2, st);
            wait_vm<2 * NDMA>();
        } else if (RESHAPE && !more && r_st < 0) {
            issue_r(st);
            r_st = st;
            wait_vm<NDMA_R>();
        } else {
            wait_vm<0>();
        }
        cur = nxt;
        nxt = nx2;
        st ^= 1;
    }
    if (RESHAPE && r_st < 0) {  // a block with no kept key block
        issue_r(0);
        r_st = 0;
    }
    wait_vm<0>();
    if (!RESHAPE) r_st = st;  // any stage serves as the output tile

    // ---- epilogue: O = factor * acc (+ R) into the tile in LDS, then row stores -----
    lds_u8* const Ot = lds + r_st * STAGE;
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int rl = qt * 32 + l32;  // row within the block
        const int row = row0 + rl;
        const float l_tot = pair_sum(l_run[qt]);
        float factor = 1.0f / l_tot;
        if (RESHAPE) factor *= fminf(1.0f, rho_r[qt] + a.rho_delta);
        if (STATS && hi == 0 && row < T) {
            const size_t si = (size_t)bh * T + row;
            if (a.row_max) a.row_max[si] = m_top[qt] * a.scale_nat;
            if (a.row_sum) a.row_sum[si] = l_tot * __builtin_amdgcn_exp2f((m_run[qt] - m_top[qt]) * c2);
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int d = 32 * dt + 8 * j + 4 * hi;
                if (d < D) {
                    lds_u32x2* p = (lds_u32x2*)(Ot + rl * ROWB + (((d >> 3) ^ kswz<D>(rl)) * 16) + (d & 7) * 2);
                    float y[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) y[i] = oacc[qt][dt][4 * j + i] * factor;
                    if (RESHAPE) {
                        const u32x2 r2 = *p;
                        y[0] += lo_f(r2[0]);
                        y[1] += hi_f(r2[0]);
                        y[2] += lo_f(r2[1]);
                        y[3] += hi_f(r2[1]);
                    }
                    *p = u32x2{pack_bf16(y[0], y[1]), pack_bf16(y[2], y[3])};
                }
            }
        }
    }
    // rows leave as 16-byte stores
    for (int u = lane; u < BS * DC; u += 64) {
        const int rl = u / DC, ch = u - (u / DC) * DC;
        const int row = row0 + rl;
        if (row >= T) continue;
        const u32x4 v = *(const lds_u32x4*)(Ot + rl * ROWB + ((ch ^ kswz<D>(rl)) * 16));
        *reinterpret_cast<u32x4*>(a.o + head_off + (size_t)row * D + 8 * ch) = v;
    }
}

template <int D, int BS, bool RESHAPE, bool STATS>
hipError_t launch_one(const AttnArgs& a, hipStream_t stream) {
    dim3 grid(8 * a.per_xcd), block(64);
    hipLaunchKernelGGL((attn_fwd<D, BS, RESHAPE, STATS>), grid, block, 0, stream, a);
    return hipGetLastError();
}

template <int D, int BS>
hipError_t launch_db(const AttnArgs& a, bool reshape, hipStream_t stream) {
    const bool stats = a.row_max != nullptr || a.row_sum != nullptr;
    if (reshape) return stats ? launch_one<D, BS, true, true>(a, stream) : launch_one<D, BS, true, false>(a, stream);
    return stats ? launch_one<D, BS, false, true>(a, stream) : launch_one<D, BS, false, false>(a, stream);
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int D, int block, bool reshape, hipStream_t stream) {
    if (D == 64) return block == 64 ? launch_db<64, 64>(a, reshape, stream) : launch_db<64, 32>(a, reshape, stream);
    return block == 64 ? launch_db<72, 64>(a, reshape, stream) : launch_db<72, 32>(a, reshape, stream);
}

}  // namespace rt
