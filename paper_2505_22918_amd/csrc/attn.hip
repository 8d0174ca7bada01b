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
// K and V chunks move from HBM/L2 straight into a two-stage LDS ring with
// buffer_load ... lds (no staging registers); the DMA for chunk i+1 is in
// flight while chunk i is computed.  A buffer resource per chunk ends at the
// last key row, so rows past T arrive as zeros (their scores are then masked
// to -inf).  Rows stay row-major in LDS: K is read as the A operand with
// 16-byte reads, V^T through ds_read_b64_tr_b16, the CDNA4 LDS transpose read.
// 16-byte slots of a row are XOR-swizzled by row so both reads are free of
// bank conflicts (72-wide heads use 144-byte rows, which spread banks as is).
//
// The running max only moves when a new chunk exceeds it by more than 2^8 in
// probability units; until then exponentials are taken against the stale max
// (bounded by 2^8, exact in fp32) and the accumulator is not rescaled.  The
// true max is tracked separately and the row sum is moved to it at the end, so
// the emitted statistics are exactly max and exp-sum.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace rt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) int32_t* csr_ptr;
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr float kRescaleLog2 = 8.0f;  // stale-max slack, in log2 units

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

// K rows: 8 consecutive rows read the same slot -> XOR with r & 7.
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

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14]).
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// 16 bytes per lane from buffer `rsrc` at byte offset `voff` into LDS at
// m0 + 16 * lane (buffer_load_dwordx4 ... lds).  m0 is reserved by the compiler
// (never allocated) and is set before every use.
__device__ __forceinline__ void dma16(uint32_t lds_addr, int voff, i32x4 rsrc) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(rsrc)
        : "memory");
}

template <int D, int BS>
constexpr int kWaves = (D == 72 && BS == 64) ? 1 : 2;

template <int D, int BS, bool RESHAPE>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(kWaves<D, BS>)))
void attn_fwd(AttnArgs a) {
    using G = Geo<D>;
    constexpr int DK = G::DK;
    constexpr int DV = G::DV;
    constexpr int QT = BS / 32;              // 32-query tiles per workgroup
    constexpr int DS = DK / 16;              // k-steps of Q K^T
    constexpr int DT = DV / 32;              // 32-row tiles of O^T
    constexpr int DC = D / 8;                // 16-byte chunks per token row
    constexpr int ROWB = G::SLOTS * 16;      // LDS bytes per row
    constexpr int TILE = 32 * ROWB;          // LDS bytes per K or V chunk
    constexpr int NSLOT = 32 * G::SLOTS;     // 16-byte slots per chunk
    constexpr int NDMA = (NSLOT + 63) / 64;  // DMA instructions per chunk and tensor
    constexpr int OSTR = D + 4;              // fp32 output stage row stride
    constexpr int RING = 4 * TILE + 256;     // K0 K1 V0 V1 + slack for padded V^T reads
    constexpr int OST = 32 * OSTR * 4;
    constexpr int SMEM = RING > OST ? RING : OST;

    __shared__ __attribute__((aligned(1024))) unsigned char smem[SMEM];
    lds_u8* const lds = (lds_u8*)smem;

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

    // ---- Q^T operands: lane holds query l32 of tile qt, head dims 16s + 8hi .. +7
    bf16x8 qop[QT][DS];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        int row = qb * BS + qt * 32 + l32;
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
    // the first 64 column indices live in one VGPR (lane i holds entry e_beg + i);
    // longer rows read the rest with scalar loads
    int cols = -1;
    if (!a.dense && lane < e_end - e_beg) cols = a.col_idx[e_beg + lane];
    int e = e_beg, c = 0;
    auto next_chunk = [&]() -> int {
        while (e < e_end) {
            int kb;
            if (a.dense) {
                kb = e;
            } else if (e - e_beg < 64) {
                kb = __builtin_amdgcn_readlane(cols, e - e_beg);
            } else {
                kb = ((csr_ptr)a.col_idx)[e];
            }
            if (kb >= 0 && kb < a.n_blk && c < BS / 32) {
                const int base = kb * BS + 32 * c;
                if (base < T) {
                    ++c;
                    return base;
                }
            }
            ++e;
            c = 0;
        }
        return -1;
    };

    // DMA of the 32-key chunk starting at key `base` into ring stage `st`.  The
    // buffer resource ends at row T, so rows past it read as zeros.  The loads are
    // issued from inline assembly: the compiler then neither orders them against
    // the LDS reads of the other stage nor waits for them; the loop waits on the
    // vector-memory counter itself.
    auto issue = [&](int base, int st) {
        const int64_t left = (int64_t)(T - base) * (D * 2);
        const int nrec = left < (int64_t)(32 * D * 2) ? (int)left : 32 * D * 2;
        const uint64_t kp = (uint64_t)(uintptr_t)(Kh + (size_t)base * D);
        const uint64_t vp = (uint64_t)(uintptr_t)(Vh + (size_t)base * D);
        const i32x4 kr = {(int)(uint32_t)kp, (int)((uint32_t)(kp >> 32) & 0xffffu), nrec, 0x00020000};
        const i32x4 vr = {(int)(uint32_t)vp, (int)((uint32_t)(vp >> 32) & 0xffffu), nrec, 0x00020000};
        const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
#pragma unroll
        for (int n = 0; n < NDMA; ++n) {
            if (NSLOT % 64 == 0 || n * 64 + lane < NSLOT)
                dma16(lds0 + st * TILE + n * 1024, kdma[n], kr);
        }
#pragma unroll
        for (int n = 0; n < NDMA; ++n) {
            if (NSLOT % 64 == 0 || n * 64 + lane < NSLOT)
                dma16(lds0 + (2 + st) * TILE + n * 1024, vdma[n], vr);
        }
    };

    const float c2 = a.scale_log2;  // log2(e) / sqrt(D)
    f32x16 oacc[QT][DT];
    float m_run[QT], m_top[QT], l_run[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        m_run[qt] = -INFINITY;
        m_top[qt] = -INFINITY;
        l_run[qt] = 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[qt][dt] = f32x16{};
    }

    wait_vm<0>();  // Q operands and the CSR window are in registers
    int cur = next_chunk();
    if (cur >= 0) issue(cur, 0);
    int nxt = next_chunk();
    int st = 0;
    while (cur >= 0) {
        if (nxt >= 0) {
            issue(nxt, st ^ 1);
            wait_vm<2 * NDMA>();
        } else {
            wait_vm<0>();
        }
        lds_u8* const Ks = lds + st * TILE;
        lds_u8* const Vs = lds + (2 + st) * TILE;

        // S^T = K Q^T
        f32x16 sacc[QT];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) sacc[qt] = f32x16{};
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            const bf16x8 kop = *(lds_bf16x8*)(Ks + k_rd[s]);
#pragma unroll
            for (int qt = 0; qt < QT; ++qt)
                sacc[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[qt][s], sacc[qt], 0, 0, 0);
        }

        // online softmax; lane holds keys cur + 8j + 4hi + i for acc index 4j + i
        const bool tail = cur + 32 > T;
        bf16x8 pop[QT][2];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            if (tail) {
#pragma unroll
                for (int x = 0; x < 16; ++x) {
                    const int key = cur + 8 * (x >> 2) + 4 * hi + (x & 3);
                    if (key >= T) sacc[qt][x] = -INFINITY;
                }
            }
            float mx = fmaxf(fmaxf(sacc[qt][0], sacc[qt][1]), sacc[qt][2]);
#pragma unroll
            for (int x = 3; x < 15; x += 2) mx = fmaxf(fmaxf(mx, sacc[qt][x]), sacc[qt][x + 1]);
            mx = fmaxf(mx, sacc[qt][15]);
            mx = pair_max(mx);
            m_top[qt] = fmaxf(m_top[qt], mx);
            const bool need = (mx - m_run[qt]) * c2 > kRescaleLog2;
            if (__builtin_amdgcn_ballot_w64(need)) {
                const float mnew = need ? mx : m_run[qt];
                const float alpha = __builtin_amdgcn_exp2f((m_run[qt] - mnew) * c2);
                l_run[qt] *= alpha;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) oacc[qt][dt] *= alpha;
                m_run[qt] = mnew;
            }
            const float mc = m_run[qt] * c2;
            float lsum = 0.f;
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
                for (int x = 0; x < 8; ++x) {
                    const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[qt][8 * ks + x], c2, -mc));
                    lsum += p;
                    pop[qt][ks][x] = (__bf16)p;
                }
            }
            l_run[qt] += lsum;
        }

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

        cur = nxt;
        nxt = next_chunk();
        st ^= 1;
    }

    // ---- epilogue, one 32-query tile at a time through an fp32 LDS stage ------------
    float* Os = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int row = qb * BS + qt * 32 + l32;
        const float l_tot = pair_sum(l_run[qt]);
        float factor = 1.0f / l_tot;
        if (RESHAPE) {
            const float r = (row < T ? a.rho[(size_t)bh * T + row] : 0.f) + a.rho_delta;
            factor *= fminf(1.0f, r);
        }
        if (hi == 0 && row < T) {
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
                    f32x4 v4;
#pragma unroll
                    for (int i = 0; i < 4; ++i) v4[i] = oacc[qt][dt][4 * j + i] * factor;
                    *reinterpret_cast<f32x4*>(Os + l32 * OSTR + d) = v4;
                }
            }
        }
        // rows back out as 16-byte bf16 stores (plus the residual)
        for (int u = lane; u < 32 * DC; u += 64) {
            const int r = u / DC, ch = u - (u / DC) * DC;
            const int orow = qb * BS + qt * 32 + r;
            if (orow >= T) continue;
            const f32x4 x0 = *reinterpret_cast<const f32x4*>(Os + r * OSTR + 8 * ch);
            const f32x4 x1 = *reinterpret_cast<const f32x4*>(Os + r * OSTR + 8 * ch + 4);
            float y[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
            const size_t off = head_off + (size_t)orow * D + 8 * ch;
            if (RESHAPE) {
                const u32x4 rv = *reinterpret_cast<const u32x4*>(a.resid + off);
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    y[2 * w] += bf16_to_f32(rv[w] & 0xffffu);
                    y[2 * w + 1] += bf16_to_f32(rv[w] >> 16);
                }
            }
            bf16x8 ob;
#pragma unroll
            for (int i = 0; i < 8; ++i) ob[i] = (__bf16)y[i];
            *reinterpret_cast<bf16x8*>(a.o + off) = ob;
        }
    }
}

template <int D, int BS, bool RESHAPE>
hipError_t launch_one(const AttnArgs& a, hipStream_t stream) {
    dim3 grid(8 * a.per_xcd), block(64);
    hipLaunchKernelGGL((attn_fwd<D, BS, RESHAPE>), grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int D, int block, bool reshape, hipStream_t stream) {
    if (D == 64) {
        if (block == 64) return reshape ? launch_one<64, 64, true>(a, stream) : launch_one<64, 64, false>(a, stream);
        return reshape ? launch_one<64, 32, true>(a, stream) : launch_one<64, 32, false>(a, stream);
    }
    if (block == 64) return reshape ? launch_one<72, 64, true>(a, stream) : launch_one<72, 64, false>(a, stream);
    return reshape ? launch_one<72, 32, true>(a, stream) : launch_one<72, 32, false>(a, stream);
}

}  // namespace rt
