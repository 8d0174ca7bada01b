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
// never leaves registers.  The rows of the V^T operand are permuted so that
// each lane's 16 accumulator values of O^T are 16 consecutive head dims of
// its query: a lane reads its residual values with 16-byte LDS reads and
// stores its output rows with 16-byte stores straight from registers.
//
// Memory.  Q arrives by buffer loads straight into its B-operand registers.
// K and V chunks move from HBM/L2 into LDS rings (three K stages, two V stages,
// 20 KB per wave at D = 64) with buffer_load ... lds (no staging registers);
// K(t+2), K(t+3) and V(t+1) are in flight while chunk t is softmaxed.  Buffer
// resources end at the last key row, so rows past T arrive as zeros (their
// scores are then masked).
// Rows stay row-major in LDS: K is read as the A operand with 16-byte reads,
// V^T through ds_read_b64_tr_b16, the CDNA4 LDS transpose read.  16-byte slots
// of a row are XOR-swizzled by row to spread both reads over the banks (72-wide
// heads use 144-byte rows, which spread banks as is).
//
// Software pipeline.  Step t issues the DMA of K(t+3), runs the P V product of
// chunk t-1 on the matrix cores under the exponentials of chunk t's softmax,
// issues the DMA of V(t+1) into the stage V(t-1) has just left, packs chunk t's
// probabilities to bf16 in the registers P V(t-1) has just read, and computes
// S(t+1) = K Q^T into the registers softmax(t) has just read (no register
// copies between steps).  The last step has no S product.  In the fused
// reshape the K loads of the two chunks past the row, which would only read
// zeros, bring the block's residual rows into their K stages instead, two to
// three steps before the epilogue reads them.
//
// Softmax.  The running max starts at the first chunk's max and moves only
// when a chunk's probabilities against it reach 2^64 (far below fp32 and bf16
// overflow); that rare case rescales O and l and recomputes the chunk.
// Without requested statistics no per-chunk max is taken: the overflow test
// reads the chunk's row sum, which then adds the bf16 probabilities P V uses.
// With statistics the exact max is tracked and l, summed in fp32, is moved to
// it at the end, so the emitted pair is exactly max and exp-sum.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kernels.h"

namespace rt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) int32_t* csr_ptr;
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

constexpr float kJump = 18446744073709551616.0f;  // 2^64: stale-max limit on a probability
constexpr int kOob = 0x40000000;                   // buffer offset past every record: reads zero

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
// V rows: a transpose read covers 4 consecutive rows and, per row, the two
// slots s and s ^ 2 -> XOR with {0, 1, 4, 5}[r & 3] keeps the 8 (row, slot)
// pairs of a half-wave on distinct banks.
template <int D>
__device__ __forceinline__ int vswz(int r) {
    return Geo<D>::SWZ ? (((r & 2) << 1) | (r & 1)) : 0;
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
    const bf16x2 v = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, v);
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
// (never allocated) and is set before every use; this is sound only while the
// compiled code keeps nothing else in m0, which the tests check on the
// assembly of every build.  Issued from inline assembly so
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

// Four such loads at byte offsets voff + 1024 n into LDS m0 + 1024 n + 16 * lane,
// n = 0..3: the instruction offset moves both the source and the LDS destination.
__device__ __forceinline__ void dma16x4(uint32_t lds_addr, int voff, i32x4 rsrc) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen offset:1024 lds\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen offset:2048 lds\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen offset:3072 lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(rsrc)
        : "memory");
}

// 16 bytes per lane from buffer `rsrc` at byte offset `voff` into registers.
// The data lands later: the caller waits on the vector-memory counter and
// then passes the value through settle() before reading it.
__device__ __forceinline__ u32x4 vload16(int voff, i32x4 rsrc) {
    u32x4 v;
    asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen" : "=&v"(v) : "v"(voff), "s"(rsrc) : "memory");
    return v;
}
__device__ __forceinline__ void settle(u32x4& v) { asm volatile("" : "+v"(v)); }

__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, int bytes) {
    const uint64_t p = (uint64_t)(uintptr_t)base;
    return i32x4{(int)(uint32_t)p, (int)((uint32_t)(p >> 32) & 0xffffu), bytes, 0x00020000};
}

template <int D, int BS>
constexpr int kWaves = (D == 72 && BS == 64) ? 1 : 2;

template <int D, int BS, bool RESHAPE, bool STATS, bool CACHE>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(kWaves<D, BS>)))
void attn_fwd(AttnArgs a) {
    using G = Geo<D>;
    constexpr int DK = G::DK;
    constexpr int DV = G::DV;
    constexpr int QT = BS / 32;              // 32-query tiles per workgroup
    constexpr int DS = DK / 16;              // k-steps of Q K^T
    constexpr int DT = DV / 32;              // 32-row tiles of O^T
    constexpr int DC = D / 8;                // 16-byte chunks per token row
    constexpr int ROWB = G::SLOTS * 16;      // LDS bytes per K / V row (= 2 * D)
    constexpr int TILE = 32 * ROWB;          // LDS bytes per K or V chunk
    constexpr int NSLOT = 32 * G::SLOTS;     // 16-byte slots per chunk and tensor
    constexpr int NDMA = (NSLOT + 63) / 64;  // DMA instructions per chunk and tensor
    // three K stages and two V stages (+ slack for the padded V^T reads of a 72-wide
    // head): 20 KB per wave at D = 64, so 8 waves fill a CU's 160 KB
    constexpr int SMEM = 5 * TILE + (D == 64 ? 0 : 256);
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
    const int nrow = (T - row0) < BS ? (T - row0) : BS;

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
    // V^T A-operand transpose reads.  In a group of 16 lanes (G4 = lane / 16),
    // lane L supplies key row 4*hi + L/4 (+16ks, +8 for the second read) at the
    // 4 head dims starting at 32dt + 16(L & 1) + 8(G4 & 1) + 4((L >> 1) & 1).
    // Lane 4a + b of the group then receives 4 consecutive keys of head dim
    // 32dt + 16(a & 1) + 8(G4 & 1) + 4(a >> 1) + b, which puts head dim
    // 32dt + 16h + 4j + i on O^T accumulator row 8j + 4h + i: lane (h, col)
    // accumulates head dims 32dt + 16h .. +15 of query col.
    int v_rd[DT];
    {
        const int G4 = lane >> 4, L = lane & 15;
        const int r = 4 * hi + (L >> 2);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const int d = 32 * dt + 16 * (L & 1) + 8 * (G4 & 1) + 4 * ((L >> 1) & 1);
            v_rd[dt] = r * ROWB + (((d >> 3) ^ vswz<D>(r)) * 16) + (d & 7) * 2;
        }
    }
    // rows of this block in Q / R / O; rows past T read as zeros
    const i32x4 q_rs = buffer_rsrc(a.q + head_off + (size_t)row0 * D, nrow * D * 2);
    // Q^T operands: lane holds query l32 of tile qt, head dims 16s + 8hi .. +7
    // (zero past D and past T).  Issued first, so that their HBM latency runs
    // under the reads of the CSR row below.
    u32x4 qraw[QT][DS];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            const int ch = 2 * s + hi;
            qraw[qt][s] = vload16(ch < DC ? (qt * 32 + l32) * (D * 2) + ch * 16 : kOob, q_rs);
        }
    }

    // ---- kept key blocks of this query block ----------------------------------------
    int e_beg, e_end;
    if (a.dense) {
        e_beg = 0;
        e_end = a.n_blk;
    } else {
        // the mask of this (batch, head): shared, per head, or per (batch, head)
        const int mid = a.n_masks <= 1 ? 0 : (a.n_masks == a.heads ? bh % a.heads : bh);
        const csr_ptr rp = (csr_ptr)a.row_ptr + (size_t)mid * (a.n_blk + 1);
        e_beg = rp[qb];
        e_end = rp[qb + 1];
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
    wait_vm<0>();
    asm volatile("" : "+v"(cols));  // the load has landed; later reads need no wait
    // The caching step walks every key block: the kept ones first (chunks
    // 0 .. n_in-1, CSR order), then the others in ascending order.
    const int n_in = (e_end - e_beg) * (BS / 32);
    const int n_chunk = CACHE ? a.n_blk * (BS / 32) : n_in;
    auto kept_at = [&](int j) -> int {  // entry e_beg + j of the CSR row
        return j < 64 ? __builtin_amdgcn_readlane(cols, j) : ((csr_ptr)a.col_idx)[e_beg + j];
    };
    int gen_kb = -1, gen_e = 0;  // complement walk: last block emitted, next kept entry
    // A chunk is addressed by the byte offset of its first key row in the head's
    // K (or V) buffer, base * 2D, or kOob for a chunk that holds no key.
    // Except in the caching walk, the offsets of 64 consecutive chunks tb ..
    // tb+63 sit in one VGPR, lane i holding chunk tb + i (kOob past the row): a
    // step reads the chunk it loads with one v_readlane and tests no bounds; the
    // walk refills the table every 64 steps.  The caching walk computes offsets
    // with scalar code.
    int tab = kOob, tb = 0;
    auto fill_tab = [&](int c0) {
        tb = c0;
        const int i = c0 + lane;
        const int j = i / (BS / 32), half = i - j * (BS / 32);
        int kb = j;
        if (!a.dense) {
            const int last = (c0 + 63 < n_chunk ? c0 + 63 : n_chunk - 1) / (BS / 32);
            if (last < 64) {  // every entry this table needs sits in `cols`
                kb = __builtin_amdgcn_ds_bpermute((j & 63) << 2, cols);
            } else {  // a row of more than 64 entries: read them (rare; drains the loads)
                const int e = i < n_chunk ? e_beg + j : 0;
                kb = ((const int32_t*)a.col_idx)[e];
                wait_vm<0>();
            }
        }
        const int base = kb * BS + 32 * half;
        tab = (i < n_chunk && kb >= 0 && kb < a.n_blk && base < T) ? base * (D * 2) : kOob;
    };
    if (!CACHE) fill_tab(0);
    // Offset of chunk i by scalar code.  Called for i = 0, 1, 2, ... in order,
    // once each (the complement walk relies on it).
    auto chunk_off = [&](int i) -> int {
        int kb, half;
        if (CACHE && i >= n_in) {
            const int jc = (i - n_in) / (BS / 32);
            half = (i - n_in) - jc * (BS / 32);
            if (half == 0) {
                int c = gen_kb + 1;
                while (gen_e < e_end - e_beg) {  // skip the kept blocks (sorted ascending)
                    const int kk = kept_at(gen_e);
                    if (kk < c) {
                        ++gen_e;
                    } else if (kk == c) {
                        ++c;
                        ++gen_e;
                    } else {
                        break;
                    }
                }
                gen_kb = c;
            }
            kb = gen_kb;
        } else {
            const int j = i / (BS / 32);
            half = i - j * (BS / 32);
            kb = a.dense ? j : kept_at(j);
        }
        const int base = kb * BS + 32 * half;
        return (kb >= 0 && kb < a.n_blk && base < T) ? base * (D * 2) : kOob;
    };
    // offset of one of the first three chunks
    auto first_off = [&](int i) -> int {
        if (CACHE) return i < n_chunk ? chunk_off(i) : kOob;
        return __builtin_amdgcn_readlane(tab, i);
    };

    // LDS map: K(t) in stage t % 3 at [0, 3 TILE), V(t) in stage t % 2 at
    // [3 TILE, 5 TILE).
    auto k_off = [&](int st) { return st * TILE; };
    auto v_off = [&](int st) { return (3 + st) * TILE; };

    // DMA of the 32-key chunk at byte offset `boff` of a head's K or V (buffer
    // resource `rs`: the whole head, T rows) to LDS byte offset `dst`.  Rows past
    // T fall outside the buffer and read as zeros; a chunk that holds no key
    // (kOob) lies past the buffer, so its loads read zeros and touch no memory.
    // Every call issues NDMA loads, so all waits below are constants.
    const i32x4 k_rs = buffer_rsrc(Kh, T * D * 2);
    const i32x4 v_rs = buffer_rsrc(Vh, T * D * 2);
    auto issue = [&](const i32x4& rs, const int (&off)[NDMA], int boff, int dst) {
        if (NSLOT == 4 * 64) {
            dma16x4(lds0 + dst, off[0] + boff, rs);
        } else {
#pragma unroll
            for (int n = 0; n < NDMA; ++n) {
                if (NSLOT % 64 == 0 || n * 64 + lane < NSLOT) dma16(lds0 + dst + n * 1024, off[n] + boff, rs);
            }
        }
    };
    // K load of chunk c into LDS byte offset dst.  In the fused reshape the loads
    // of chunks n_chunk .. n_chunk + QT - 1, which lie past the row and would only
    // fill their stages with zeros, instead bring the block's residual rows
    // 32j .. 32j + 31 (j = c - n_chunk) in the K layout: R lands two to three steps
    // before the epilogue reads it, with the same number of loads per step.
    const i32x4 r_rs = RESHAPE ? buffer_rsrc(a.resid + head_off + (size_t)row0 * D, nrow * D * 2) : k_rs;
    auto issue_k = [&](int c, int boff, int dst) {
        if (RESHAPE) {
            const int rj = c - n_chunk;
            if (rj >= 0 && rj < QT) {
                issue(r_rs, kdma, rj * 32 * (D * 2), dst);
                return;
            }
        }
        issue(k_rs, kdma, boff, dst);
    };

    // ---- prologue ---------------------------------------------------------------------
    float rho_r[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int row = row0 + qt * 32 + l32;
        rho_r[qt] = (RESHAPE && a.rho && row < T) ? a.rho[(size_t)bh * T + row] : 0.f;
    }
    const int c0 = first_off(0);
    const int c1 = first_off(1);
    const int c2b = first_off(2);
    // issue order Q, K(0), V(0), K(1), K(2); afterwards step t issues K(t+3) at its
    // start and V(t+1) after its P V product, so waiting for V(t-1) at the start of
    // step t leaves exactly three chunk loads (K(t+2), V(t), K(t+3)) in flight
    issue_k(0, c0, k_off(0));
    issue(v_rs, vdma, c0, v_off(0));
    issue_k(1, c1, k_off(1));
    issue_k(2, c2b, k_off(2));
    wait_vm<3 * NDMA>();  // Q and K(0) have landed
    bf16x8 qop[QT][DS];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            settle(qraw[qt][s]);
            qop[qt][s] = __builtin_bit_cast(bf16x8, qraw[qt][s]);
        }
    }

    const float c2 = a.scale_log2;  // log2(e) / sqrt(D)
    f32x16 oacc[QT][DT];
    float m_run[QT], m_top[QT], l_run[QT];
    float l_in[QT];  // caching step: kept-block exp-sum against m_run, once the kept walk is done
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        m_run[qt] = -1e30f;  // finite: a fully masked chunk then yields p = 0, not NaN
        m_top[qt] = -INFINITY;
        l_run[qt] = 0.f;
        l_in[qt] = 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[qt][dt] = f32x16{};
    }

    // S^T = K Q^T for the K chunk at LDS byte offset `ko`
    auto qk = [&](int ko, f32x16 (&sc)[QT]) {
        const lds_u8* Ks = lds + ko;
        bf16x8 kop[DS];
#pragma unroll
        for (int s = 0; s < DS; ++s) kop[s] = *(const lds_bf16x8*)(Ks + k_rd[s]);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) sc[qt] = f32x16{};
#pragma unroll
        for (int s = 0; s < DS; ++s) {
#pragma unroll
            for (int qt = 0; qt < QT; ++qt)
                sc[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[s], qop[qt][s], sc[qt], 0, 0, 0);
        }
    };
    // keys past T, or a chunk holding no key, score -inf.  Chunks at offsets up to
    // full_lim hold 32 keys below T (kOob lies above every such offset).
    const int full_lim = (T - 32) * (D * 2);
    auto mask = [&](int boff, f32x16 (&sc)[QT]) {
        if (boff <= full_lim) return;
        const int base = boff == kOob ? -1 : boff / (D * 2);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
            for (int x = 0; x < 16; ++x) {
                const int key = base + 8 * (x >> 2) + 4 * hi + (x & 3);
                if (base < 0 || key >= T) sc[qt][x] = -INFINITY;
            }
        }
    };
    // V^T operand of k-step ks of the V chunk at LDS byte offset `vo`: two
    // transpose reads of 4 key rows each
    auto v_operand = [&](int vo, int dt, int ks) -> bf16x8 {
        const lds_u8* Vs = lds + vo;
        const bf16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(Vs + v_rd[dt] + 16 * ks * ROWB));
        const bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(Vs + v_rd[dt] + (16 * ks + 8) * ROWB));
        return __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
    };
    // O^T += V^T P^T for the V chunk at LDS byte offset `vo`
    auto pv = [&](int vo, const bf16x8 (&pp)[QT][2]) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x8 vv = v_operand(vo, dt, ks);
#pragma unroll
                for (int qt = 0; qt < QT; ++qt)
                    oacc[qt][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vv, pp[qt][ks], oacc[qt][dt], 0, 0, 0);
            }
        }
    };
    // Row sums.  Where l only normalises O (no statistics, no caching split), l
    // sums the bf16 probabilities that P V multiplies, two per v_dot2_f32_bf16 on
    // the packed operands; numerator and denominator then use the same weights.
    // Where l, m or rho are outputs, l sums the fp32 probabilities.
    constexpr bool BF16_SUM = !STATS && !CACHE;
    // fp32 probabilities of scores x0 .. x0+3 against the running max (mc = m * c2);
    // their sum starts (first) or joins acc (fp32 row sums only)
    auto exps4 = [&](const f32x16& sc, int x0, float mc, float* p, float& acc, bool first) {
#pragma unroll
        for (int x = 0; x < 4; ++x) p[x] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[x0 + x], c2, -mc));
        if (!BF16_SUM) {
            const float part = (p[0] + p[1]) + (p[2] + p[3]);
            acc = first ? part : acc + part;
        }
    };
    // sum of the 16 bf16 probabilities packed in pk (two partial chains)
    auto bf16_sum = [&](const bf16x8 (&pk)[2]) -> float {
        const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
        float a0 = 0.f, a1 = 0.f;
        a0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pk[0], pk[0], 0, 1), one2, a0, false);
        a1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pk[1], pk[1], 0, 1), one2, a1, false);
        a0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pk[0], pk[0], 2, 3), one2, a0, false);
        a1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pk[1], pk[1], 2, 3), one2, a1, false);
        a0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pk[0], pk[0], 4, 5), one2, a0, false);
        a1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pk[1], pk[1], 4, 5), one2, a1, false);
        a0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pk[0], pk[0], 6, 7), one2, a0, false);
        a1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pk[1], pk[1], 6, 7), one2, a1, false);
        return a0 + a1;
    };
    // all 16 probabilities of tile qt; returns their sum
    auto exps16 = [&](const f32x16& sc, float mc, float (&p)[16]) -> float {
        float s0 = 0.f, s1 = 0.f;
        exps4(sc, 0, mc, p + 0, s0, true);
        exps4(sc, 4, mc, p + 4, s1, true);
        exps4(sc, 8, mc, p + 8, s0, false);
        exps4(sc, 12, mc, p + 12, s1, false);
        return s0 + s1;
    };
    // bf16 B operands of the P V product: keys 0-7 and 8-15 of the lane's 16
    auto pack16 = [&](const float (&p)[16], bf16x8 (&pk)[2]) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const bf16x2 a0 = {(__bf16)p[8 * h + 0], (__bf16)p[8 * h + 1]};
            const bf16x2 a1 = {(__bf16)p[8 * h + 2], (__bf16)p[8 * h + 3]};
            const bf16x2 a2 = {(__bf16)p[8 * h + 4], (__bf16)p[8 * h + 5]};
            const bf16x2 a3 = {(__bf16)p[8 * h + 6], (__bf16)p[8 * h + 7]};
            const bf16x4 lo = __builtin_shufflevector(a0, a1, 0, 1, 2, 3);
            const bf16x4 hi4 = __builtin_shufflevector(a2, a3, 0, 1, 2, 3);
            pk[h] = __builtin_shufflevector(lo, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
        }
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

    // Caching step, end of the kept walk: O_s = acc / l goes to the output rows
    // (read back by the epilogue), l becomes l_in, and the walk over the other
    // blocks starts a fresh sum and accumulator against the same running max.
    auto flush_kept = [&]() {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            const int row = row0 + qt * 32 + l32;
            const float inv = 1.0f / pair_sum(l_run[qt]);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int ch = 4 * dt + 2 * hi + u;
                    if (ch < DC && row < T) {
                        const f32x16& acc = oacc[qt][dt];
                        const u32x4 o4 = {pack_bf16(acc[8 * u + 0] * inv, acc[8 * u + 1] * inv),
                                          pack_bf16(acc[8 * u + 2] * inv, acc[8 * u + 3] * inv),
                                          pack_bf16(acc[8 * u + 4] * inv, acc[8 * u + 5] * inv),
                                          pack_bf16(acc[8 * u + 6] * inv, acc[8 * u + 7] * inv)};
                        *reinterpret_cast<u32x4*>(a.o + head_off + (size_t)row * D + 8 * ch) = o4;
                    }
                }
            }
            l_in[qt] = l_run[qt];
            l_run[qt] = 0.f;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) oacc[qt][dt] = f32x16{};
        }
    };

    // ---- software pipeline over chunks 0 .. n-1 -----------------------------------
    // s holds the scores of the chunk being softmaxed, pk the bf16 probabilities of
    // the chunk before it; both are updated in place each step.
    f32x16 s[QT];
    bf16x8 pk[QT][2];
    if (n_chunk > 0) {
        qk(0, s);
        mask(c0, s);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) m_run[qt] = fmaxf(chunk_max(s[qt]), -1e30f);
    }
    // rolling window of chunk offsets b_t = off(t), b_t1, b_t2; LDS byte offsets
    // of the stages of K(t) (k3) and of V(t) (vo), which moves between the two V
    // stages by xor with vtog
    int b_t = c0, b_t1 = c1, b_t2 = c2b;
    int k3 = k_off(0);
    int vo = v_off(0);
    constexpr int vtog = (3 * TILE) ^ (4 * TILE);

    // Step t: issue K(t+3) (HAS_QK) and wait for K(t+1) and V(t-1).  Then
    //   A: P V(t-1) (HAS_PV) on the matrix cores, interleaved with the
    //      exponentials and row sums of softmax(t) in fp32; then the DMA of
    //      V(t+1) into the stage V(t-1) occupied;
    //   the rare rescale (a probability reached 2^64: O and l move to the new
    //      max, chunk t is recomputed; P V(t-1) is in O by then);
    //   B: chunk t's bf16 probabilities into pk (P V(t-1) has read it), then
    //      S(t+1) = K Q^T (HAS_QK) into s (softmax(t) has read it).
    // The step without S product is the last one.
    auto step = [&](int t, auto has_qk, auto has_pv) {
        constexpr bool HAS_QK = decltype(has_qk)::value;
        constexpr bool HAS_PV = decltype(has_pv)::value;
        const int vp = vo ^ vtog;                           // stage of V(t-1) and V(t+1)
        const int kn = k3 == 2 * TILE ? 0 : k3 + TILE;      // stage of K(t+1)
        int cn3 = kOob;
        if (HAS_QK) {
            if (!CACHE) {
                cn3 = __builtin_amdgcn_readlane(tab, t + 3 - tb);  // kOob past the row
            } else {
                cn3 = t + 3 < n_chunk ? chunk_off(t + 3) : kOob;
            }
            issue_k(t + 3, cn3, k3);  // K(t) was read in step t-1
        }
        if (HAS_QK && HAS_PV) {
            wait_vm<3 * NDMA>();  // K(t+2), V(t), K(t+3) may still fly
        } else if (HAS_QK || HAS_PV) {
            wait_vm<2 * NDMA>();  // step 0: K(2), K(3); last step: K(t+2), V(t)
        }

        bf16x8 vop[DT][2];
        if (HAS_PV) {
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) vop[dt][ks] = v_operand(vp, dt, ks);
            }
        }
        bf16x8 kop[DS];
        if (HAS_QK) {
            const lds_u8* Ks = lds + kn;
#pragma unroll
            for (int ss = 0; ss < DS; ++ss) kop[ss] = *(const lds_bf16x8*)(Ks + k_rd[ss]);
        }
        float mx[QT];
        if (STATS) {
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
                mx[qt] = chunk_max(s[qt]);
                m_top[qt] = fmaxf(m_top[qt], mx[qt]);
            }
        }
        // A: P V pairs, each followed by its share of the 4 x QT groups of 4
        // exponentials
        float pf[QT][16];
        float sa[QT], sb[QT];
        {
            constexpr int NA = HAS_PV ? 2 * DT : 0;
            constexpr int SLOTS = NA > 0 ? NA : 1;
            constexpr int NQ = 4 * QT;
#pragma unroll
            for (int k = 0; k < SLOTS; ++k) {
                __builtin_amdgcn_sched_barrier(0);
                if (k < NA) {
                    const int dt = k >> 1, ks = k & 1;
#pragma unroll
                    for (int qt = 0; qt < QT; ++qt)
                        oacc[qt][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[dt][ks], pk[qt][ks], oacc[qt][dt], 0, 0, 0);
                }
#pragma unroll
                for (int q = 0; q < NQ; ++q) {
                    if (q * SLOTS / NQ == k) {
                        const int qt = q / 4, part = q % 4;
                        exps4(s[qt], 4 * part, m_run[qt] * c2, pf[qt] + 4 * part, (part & 1) ? sb[qt] : sa[qt], part < 2);
                    }
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // V(t+1) into the stage P V(t-1) has just read: V gets a step and a half of
        // lead instead of one
        if (t + 1 < n_chunk) issue(v_rs, vdma, b_t1, vp);
        if (CACHE && t == n_in && t > 0) flush_kept();  // P V of chunk n_in - 1 is in O
        // Chunk t's bf16 probabilities into pk (P V(t-1) has read it) and the row
        // sums.  With bf16 row sums the S(t+1) product is issued here, between the
        // packs and the sums of the two tiles, rather than after the rescale test.
        constexpr bool QK_EARLY = BF16_SUM && HAS_QK;
        float lsum[QT];
        bool jump = false;
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            if (BF16_SUM) {
                pack16(pf[qt], pk[qt]);
                if (QK_EARLY) {
#pragma unroll
                    for (int ss = 0; ss < DS; ++ss)
                        s[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[ss], qop[qt][ss], ss == 0 ? f32x16{} : s[qt],
                                                                        0, 0, 0);
                }
                lsum[qt] = bf16_sum(pk[qt]);
            } else {
                lsum[qt] = sa[qt] + sb[qt];
            }
            jump |= !(lsum[qt] < kJump);
        }
        if (__builtin_amdgcn_ballot_w64(jump)) {
            // chunk t's scores
            f32x16 st[QT];
            if (QK_EARLY) {
                // s holds S(t+1) and K(t)'s stage holds K(t+3) by now: reload the
                // lane's K(t) row from memory and form S(t) again (same operands,
                // same products)
                u32x4 kr[DS];
#pragma unroll
                for (int ss = 0; ss < DS; ++ss) {
                    const int ch = 2 * ss + hi;
                    kr[ss] = vload16(b_t != kOob && ch < DC ? b_t + l32 * (D * 2) + ch * 16 : kOob, k_rs);
                }
                wait_vm<0>();
#pragma unroll
                for (int qt = 0; qt < QT; ++qt) {
                    st[qt] = f32x16{};
#pragma unroll
                    for (int ss = 0; ss < DS; ++ss) {
                        settle(kr[ss]);
                        st[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kr[ss]), qop[qt][ss],
                                                                         st[qt], 0, 0, 0);
                    }
                }
                mask(b_t, st);
            } else {
#pragma unroll
                for (int qt = 0; qt < QT; ++qt) st[qt] = s[qt];
            }
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
                if (!STATS) mx[qt] = chunk_max(st[qt]);
                const float mnew = fmaxf(m_run[qt], mx[qt]);
                const float alpha = __builtin_amdgcn_exp2f((m_run[qt] - mnew) * c2);
                l_run[qt] *= alpha;
                if (CACHE) l_in[qt] *= alpha;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) oacc[qt][dt] *= alpha;
                m_run[qt] = mnew;
                lsum[qt] = exps16(st[qt], mnew * c2, pf[qt]);
                if (BF16_SUM) {
                    pack16(pf[qt], pk[qt]);
                    lsum[qt] = bf16_sum(pk[qt]);
                }
            }
        }
        // B
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            l_run[qt] += lsum[qt];
            if (!BF16_SUM) pack16(pf[qt], pk[qt]);
        }
        if (HAS_QK) {
            if (!QK_EARLY) {
#pragma unroll
                for (int ss = 0; ss < DS; ++ss) {
#pragma unroll
                    for (int qt = 0; qt < QT; ++qt)
                        s[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[ss], qop[qt][ss], ss == 0 ? f32x16{} : s[qt],
                                                                        0, 0, 0);
                }
            }
            mask(b_t1, s);
        }
        b_t = b_t1;
        b_t1 = b_t2;
        b_t2 = cn3;
        k3 = kn;
        vo = vp;
    };

    using yes = std::true_type;
    using no = std::false_type;
    if (n_chunk == 1) {
        step(0, no{}, no{});
    } else if (n_chunk > 1) {
        if (!CACHE) fill_tab(3);  // steps 0 .. 60 load chunks 3 .. 63
        step(0, yes{}, no{});
        int t = 1;
        for (;;) {
            // steps up to tb + 60 find their chunk t + 3 in the table
            const int t_end = CACHE ? n_chunk - 1 : min(n_chunk - 1, tb + 61);
            for (; t < t_end; ++t) step(t, yes{}, yes{});
            if (t >= n_chunk - 1) break;
            fill_tab(t + 3);
        }
        step(n_chunk - 1, no{}, yes{});
    }
    wait_vm<0>();  // V(n-1) and, in the fused reshape, the residual rows
    asm volatile("" ::: "memory");  // no LDS read moves above the wait
    if (n_chunk > 0) pv(vo ^ vtog, pk);  // P V of the last chunk

    if (CACHE) {
        // ---- caching-step epilogue (App. A.3): with l_in, l_out and acc_out
        // against one running max, l_f = l_in + l_out, rho = l_in / l_f (Eq.8),
        // R = acc_out / l_f = O_f - rho O_s (Eq.10), O_f = rho O_s + R (Eq.1)
        const bool split = n_in < n_chunk;  // the other blocks were walked after a flush
        u32x4 osraw[QT][DT][2];
        if (split && n_in > 0) {  // O_s rows stored by the flush (complete: vmcnt is 0 here)
            const i32x4 rs = buffer_rsrc(a.o + head_off + (size_t)row0 * D, nrow * D * 2);
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
                    for (int u = 0; u < 2; ++u) {
                        const int ch = 4 * dt + 2 * hi + u;
                        osraw[qt][dt][u] = vload16(ch < DC ? (qt * 32 + l32) * (D * 2) + ch * 16 : kOob, rs);
                    }
                }
            }
            wait_vm<0>();
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    settle(osraw[qt][dt][0]);
                    settle(osraw[qt][dt][1]);
                }
            }
        } else {
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) osraw[qt][dt][0] = osraw[qt][dt][1] = u32x4{};
            }
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            const int row = row0 + qt * 32 + l32;
            const float li = pair_sum(split ? l_in[qt] : l_run[qt]);
            const float lo = split ? pair_sum(l_run[qt]) : 0.f;
            const float lf = li + lo;
            const float inv = 1.0f / lf;
            const float rho = split ? li / lf : 1.0f;  // exactly 1 when every block is kept
            if (hi == 0 && row < T && !a.postmask) {
                const size_t si = (size_t)bh * T + row;
                if (a.rho_out) a.rho_out[si] = rho;
                if (STATS) {
                    if (a.row_max) a.row_max[si] = m_top[qt] * a.scale_nat;
                    if (a.row_sum) a.row_sum[si] = lf * __builtin_amdgcn_exp2f((m_run[qt] - m_top[qt]) * c2);
                }
            }
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int ch = 4 * dt + 2 * hi + u;
                    if (ch < DC && row < T) {
                        const u32x4 os4 = osraw[qt][dt][u];
                        float r[8], of[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const float acc = oacc[qt][dt][8 * u + e] * inv;
                            const float osv = (e & 1) ? hi_f(os4[e >> 1]) : lo_f(os4[e >> 1]);
                            // R = O_f - rho O_s (Eq.10); without a ratio output,
                            // R = O_f - O_s (Eq.10 with rho = 1)
                            r[e] = split ? (a.rho_out ? acc : __builtin_fmaf(rho - 1.0f, osv, acc)) : 0.f;
                            if (a.postmask) {  // Eq.7: (A o M) V = rho O_s
                                of[e] = split ? rho * osv : acc;
                            } else {
                                of[e] = split ? __builtin_fmaf(rho, osv, acc) : acc;
                            }
                        }
                        const size_t off = head_off + (size_t)row * D + 8 * ch;
                        if (!a.postmask) {
                            *reinterpret_cast<u32x4*>(a.resid_out + off) =
                                u32x4{pack_bf16(r[0], r[1]), pack_bf16(r[2], r[3]), pack_bf16(r[4], r[5]),
                                      pack_bf16(r[6], r[7])};
                        }
                        *reinterpret_cast<u32x4*>(a.o + off) = u32x4{pack_bf16(of[0], of[1]), pack_bf16(of[2], of[3]),
                                                                     pack_bf16(of[4], of[5]), pack_bf16(of[6], of[7])};
                    }
                }
            }
        }
        return;
    }

    // ---- epilogue: O = factor * acc (+ R), 16-byte row stores from registers --------
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int rl = qt * 32 + l32;  // row within the block
        const int row = row0 + rl;
        const float l_tot = pair_sum(l_run[qt]);
        float factor = 1.0f / l_tot;
        // without a ratio (the ablation with the reshape removed) the sparse
        // output is added to the residual unscaled
        if (RESHAPE && a.rho) factor *= fminf(1.0f, rho_r[qt] + a.rho_delta);
        if (STATS && hi == 0 && row < T) {
            const size_t si = (size_t)bh * T + row;
            if (a.row_max) a.row_max[si] = m_top[qt] * a.scale_nat;
            if (a.row_sum) a.row_sum[si] = l_tot * __builtin_amdgcn_exp2f((m_run[qt] - m_top[qt]) * c2);
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int ch = 4 * dt + 2 * hi + u;  // head dims 8ch .. 8ch+7
                if (ch < DC && row < T) {
                    float y[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) y[e] = oacc[qt][dt][8 * u + e] * factor;
                    if (RESHAPE) {
                        // residual row rl, head dims 8ch .. 8ch+7, from the K stage
                        // of chunk n_chunk + qt
                        const lds_u8* Rs = lds + k_off((n_chunk + qt) % 3);
                        const u32x4 r4 = *(const lds_u32x4*)(Rs + l32 * ROWB + ((ch ^ kswz<D>(l32)) * 16));
#pragma unroll
                        for (int w = 0; w < 4; ++w) {
                            y[2 * w] += lo_f(r4[w]);
                            y[2 * w + 1] += hi_f(r4[w]);
                        }
                    }
                    const u32x4 o4 = {pack_bf16(y[0], y[1]), pack_bf16(y[2], y[3]), pack_bf16(y[4], y[5]),
                                      pack_bf16(y[6], y[7])};
                    *reinterpret_cast<u32x4*>(a.o + head_off + (size_t)row * D + 8 * ch) = o4;
                }
            }
        }
    }
}

template <int D, int BS, bool RESHAPE, bool STATS, bool CACHE>
hipError_t launch_one(const AttnArgs& a, hipStream_t stream) {
    dim3 grid(8 * a.per_xcd), block(64);
    hipLaunchKernelGGL((attn_fwd<D, BS, RESHAPE, STATS, CACHE>), grid, block, 0, stream, a);
    return hipGetLastError();
}

template <int D, int BS>
hipError_t launch_db(const AttnArgs& a, AttnMode mode, hipStream_t stream) {
    const bool stats = a.row_max != nullptr || a.row_sum != nullptr;
    switch (mode) {
        case kAttnReshape:
            return stats ? launch_one<D, BS, true, true, false>(a, stream) : launch_one<D, BS, true, false, false>(a, stream);
        case kAttnCache:
            return stats ? launch_one<D, BS, false, true, true>(a, stream) : launch_one<D, BS, false, false, true>(a, stream);
        default:
            return stats ? launch_one<D, BS, false, true, false>(a, stream)
                         : launch_one<D, BS, false, false, false>(a, stream);
    }
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int D, int block, AttnMode mode, hipStream_t stream) {
    if (D == 64) return block == 64 ? launch_db<64, 64>(a, mode, stream) : launch_db<64, 32>(a, mode, stream);
    return block == 64 ? launch_db<72, 64>(a, mode, stream) : launch_db<72, 32>(a, mode, stream);
}

}  // namespace rt
