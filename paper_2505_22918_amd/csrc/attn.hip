// Block-sparse / dense softmax attention with row statistics and the fused
// Re-ttention reshape epilogue, for gfx950 (CDNA4).
//
//   rt_attn_full            Eq.1 with the Eq.4 denominator, every key block
//   rt_attn_sparse          Eq.5, the kept key blocks of a block CSR
//   rt_attn_sparse_reshape  Eq.5, then Eq.9 (rho, ramped) and Eq.10 (residual)
//
// One workgroup is one wavefront that owns one query block (32 or 64 rows) of
// one (batch, head).  It walks the key blocks of its CSR row in 32-key chunks:
//
//   S^T = K_chunk Q^T          v_mfma_f32_32x32x16_bf16, keys x queries
//   online softmax             fp32, exp2 with log2(e)/sqrt(D) folded in
//   O^T += V_chunk^T P^T       v_mfma_f32_32x32x16_bf16, head-dim x queries
//
// Computing the transposed products keeps every query in one lane column: the
// 32x32 accumulator of S^T hands each lane 16 keys of one query, which are
// exactly the 8+8 key values the B operand of the P V product needs, so P
// never leaves registers.  V is stored transposed in LDS, with the keys of
// each 16-key group permuted to match that register order.  The row max needs
// one exchange between lane l and l^32 (v_permlane32_swap).
//
// The running max is only moved when a new chunk exceeds it by more than
// 2^8 in probability units; until then exponentials are taken against the
// stale max (bounded by 2^8, exact in fp32) and the accumulator is not
// rescaled.  The true max is tracked separately and the row sum is moved to it
// at the end, so the emitted statistics are exactly max and exp-sum.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace rt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kRescaleLog2 = 8.0f;  // stale-max slack, in log2 units

template <int D>
struct Head;
template <>
struct Head<64> {
    static constexpr int DK = 64;  // Q K^T contraction width (multiple of 16)
    static constexpr int DV = 64;  // rows of O^T (multiple of 32)
};
template <>
struct Head<72> {
    static constexpr int DK = 80;
    static constexpr int DV = 96;
};

__device__ __forceinline__ float pair_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Position of key k (0..31 within a chunk) in the transposed V tile: inside each
// group of 16 keys, keys 4..7 and 8..11 trade places (bits 2 and 3 swap).
__device__ __forceinline__ int vpos(int k) {
    int w = k & 15;
    return (k & 16) | (w & 3) | (((w >> 3) & 1) << 2) | (((w >> 2) & 1) << 3);
}

__device__ __forceinline__ uint32_t pack_lo(uint32_t a, uint32_t b) {
    return __builtin_amdgcn_perm(b, a, 0x05040100u);  // (a.lo16, b.lo16)
}
__device__ __forceinline__ uint32_t pack_hi(uint32_t a, uint32_t b) {
    return __builtin_amdgcn_perm(b, a, 0x07060302u);  // (a.hi16, b.hi16)
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// Waves per SIMD the register allocation is held to: two fit every shape
// without spilling except a 64-row tile of a 72-wide head, which stays at one.
template <int D, int BS>
constexpr int kWaves = (D == 72 && BS == 64) ? 1 : 2;

template <int D, int BS, bool RESHAPE>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(kWaves<D, BS>)))
void attn_fwd(AttnArgs a) {
    constexpr int DK = Head<D>::DK;
    constexpr int DV = Head<D>::DV;
    constexpr int QT = BS / 32;       // 32-query tiles per workgroup
    constexpr int DS = DK / 16;       // k-steps of Q K^T
    constexpr int DT = DV / 32;       // 32-row tiles of O^T
    constexpr int DC = D / 8;         // 16-byte chunks per token row
    constexpr int KSTR = DK + 8;      // LDS row stride of K (bf16), 16 B of padding
    constexpr int VSTR = 32 + 8;      // LDS row stride of V^T (bf16)
    constexpr int OSTR = D + 4;       // LDS row stride of the fp32 output stage
    constexpr int KU = 32 * DC;       // 16-byte K loads per chunk
    constexpr int KIT = (KU + 63) / 64;
    constexpr int VU = 8 * DC;        // (4-key group, 16-byte chunk) V loads per chunk
    constexpr int VIT = (VU + 63) / 64;
    constexpr int KV_ELEMS = 32 * KSTR + DV * VSTR;
    constexpr int O_ELEMS = 2 * 32 * OSTR;  // fp32 as pairs of bf16 slots
    constexpr int SMEM = KV_ELEMS > O_ELEMS ? KV_ELEMS : O_ELEMS;

    __shared__ __attribute__((aligned(16))) uint16_t smem[SMEM];
    uint16_t* Ks = smem;
    uint16_t* Vt = smem + 32 * KSTR;
    float* Os = reinterpret_cast<float*>(smem);

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

    // zero the padded head-dim columns of K and rows of V^T (never rewritten)
    if (DK > D) {
        for (int i = lane; i < 32 * (DK - D); i += 64) {
            int r = i / (DK - D), c = D + i % (DK - D);
            Ks[r * KSTR + c] = 0;
        }
    }
    if (DV > D) {
        for (int i = lane; i < (DV - D) * 32; i += 64) {
            Vt[(D + i / 32) * VSTR + (i % 32)] = 0;
        }
    }

    // Q^T operands: lane holds query l32 of tile qt, head dims 16s + 8hi .. +7
    bf16x8 qop[QT][DS];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        int row = qb * BS + qt * 32 + l32;
        row = row < T ? row : T - 1;
        const uint16_t* qr = a.q + head_off + (size_t)row * D;
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            int d0 = 16 * s + 8 * hi;
            if (d0 < D) {
                qop[qt][s] = *reinterpret_cast<const bf16x8*>(qr + d0);
            } else {
                qop[qt][s] = bf16x8{};
            }
        }
    }

    // kept key blocks of this query block
    int e_beg, e_end;
    if (a.dense) {
        e_beg = 0;
        e_end = a.n_blk;
    } else {
        e_beg = a.row_ptr[qb];
        e_end = a.row_ptr[qb + 1];
        e_beg = e_beg < 0 ? 0 : (e_beg > a.nnz ? a.nnz : e_beg);
        e_end = e_end < e_beg ? e_beg : (e_end > a.nnz ? a.nnz : e_end);
    }
    int e = e_beg, c = 0;
    // next 32-key chunk of the walk, or -1
    auto next_chunk = [&]() -> int {
        while (e < e_end) {
            int kb = a.dense ? e : a.col_idx[e];
            if (kb >= 0 && kb < a.n_blk && c < BS / 32) {
                int base = kb * BS + 32 * c;
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

    u32x4 kreg[KIT];
    u32x4 vreg[VIT][4];
    auto load_chunk = [&](int base) {
#pragma unroll
        for (int it = 0; it < KIT; ++it) {
            int u = lane + 64 * it;
            if (u < KU) {
                int r = u / DC, ch = u - (u / DC) * DC;
                int key = base + r;
                key = key < T ? key : T - 1;
                kreg[it] = *reinterpret_cast<const u32x4*>(Kh + (size_t)key * D + 8 * ch);
            }
        }
#pragma unroll
        for (int it = 0; it < VIT; ++it) {
            int u = lane + 64 * it;
            if (u < VU) {
                int grp = u / DC, ch = u - (u / DC) * DC;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    int key = base + 4 * grp + r;
                    key = key < T ? key : T - 1;
                    vreg[it][r] = *reinterpret_cast<const u32x4*>(Vh + (size_t)key * D + 8 * ch);
                }
            }
        }
    };
    auto store_chunk = [&]() {
#pragma unroll
        for (int it = 0; it < KIT; ++it) {
            int u = lane + 64 * it;
            if (u < KU) {
                int r = u / DC, ch = u - (u / DC) * DC;
                *reinterpret_cast<u32x4*>(Ks + r * KSTR + 8 * ch) = kreg[it];
            }
        }
#pragma unroll
        for (int it = 0; it < VIT; ++it) {
            int u = lane + 64 * it;
            if (u < VU) {
                int grp = u / DC, ch = u - (u / DC) * DC;
                int p = vpos(4 * grp);
                uint16_t* dst = Vt + (8 * ch) * VSTR + p;
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    uint2 lo, hv;
                    lo.x = pack_lo(vreg[it][0][w], vreg[it][1][w]);
                    lo.y = pack_lo(vreg[it][2][w], vreg[it][3][w]);
                    hv.x = pack_hi(vreg[it][0][w], vreg[it][1][w]);
                    hv.y = pack_hi(vreg[it][2][w], vreg[it][3][w]);
                    *reinterpret_cast<uint2*>(dst + (2 * w) * VSTR) = lo;
                    *reinterpret_cast<uint2*>(dst + (2 * w + 1) * VSTR) = hv;
                }
            }
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

    int cur = next_chunk();
    if (cur >= 0) {
        load_chunk(cur);
        store_chunk();
    }
    while (cur >= 0) {
        const int nxt = next_chunk();
        if (nxt >= 0) load_chunk(nxt);

        // S^T = K Q^T
        f32x16 sacc[QT];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) sacc[qt] = f32x16{};
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            bf16x8 kop = *reinterpret_cast<const bf16x8*>(Ks + l32 * KSTR + 16 * s + 8 * hi);
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
                    int key = cur + 8 * (x >> 2) + 4 * hi + (x & 3);
                    if (key >= T) sacc[qt][x] = -INFINITY;
                }
            }
            float mx = sacc[qt][0];
#pragma unroll
            for (int x = 1; x < 16; ++x) mx = fmaxf(mx, sacc[qt][x]);
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
                    float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[qt][8 * ks + x], c2, -mc));
                    lsum += p;
                    pop[qt][ks][x] = (__bf16)p;
                }
            }
            l_run[qt] += lsum;
        }

        // O^T += V^T P^T
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                bf16x8 vop = *reinterpret_cast<const bf16x8*>(Vt + (32 * dt + l32) * VSTR + 16 * ks + 8 * hi);
#pragma unroll
                for (int qt = 0; qt < QT; ++qt)
                    oacc[qt][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pop[qt][ks], oacc[qt][dt], 0, 0, 0);
            }
        }

        if (nxt >= 0) store_chunk();
        cur = nxt;
    }

    // epilogue, one 32-query tile at a time through an fp32 LDS stage
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int row = qb * BS + qt * 32 + l32;
        const float l_tot = pair_sum(l_run[qt]);
        float factor = 1.0f / l_tot;
        if (RESHAPE) {
            float r = (row < T ? a.rho[(size_t)bh * T + row] : 0.f) + a.rho_delta;
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
