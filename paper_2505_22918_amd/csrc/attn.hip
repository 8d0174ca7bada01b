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
    static_assert(RSLOT * 16 <= 2 * TILE, "Q / R tile fits two stages");
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
    wait_vm<0>();
    asm volatile("" : "+v"(cols));  // the load has landed; later reads need no wait
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

    // LDS map: K stages at [0, TILE) and [TILE, 2 TILE), V stages at [2 TILE, 3 TILE)
    // and [3 TILE, 4 TILE).  Before the walk the Q tile sits in the V stages; after
    // the last K chunk has been read the residual / output tile takes the K stages.
    auto k_off = [&](int st) { return st * TILE; };
    auto v_off = [&](int st) { return (2 + st) * TILE; };

    // DMA of the 32-key chunk of `head` starting at key `base` to LDS byte offset
    // `dst`; the buffer ends at row T, so rows past it read as zeros.  A chunk that
    // holds no key (base < 0) is not loaded.
    auto issue = [&](const uint16_t* head, const int (&off)[NDMA], int base, int dst) {
        if (base < 0) return;
        const int left = (T - base) * (D * 2);
        const int nrec = left < 32 * D * 2 ? left : 32 * D * 2;
        const i32x4 rs = buffer_rsrc(head + (size_t)base * D, nrec);
#pragma unroll
        for (int n = 0; n < NDMA; ++n) {
            if (NSLOT % 64 == 0 || n * 64 + lane < NSLOT) dma16(lds0 + dst + n * 1024, off[n], rs);
        }
    };
    // DMA of the block's BS rows of `tensor` (Q or R) to LDS byte offset `dst`, same
    // row layout and swizzle as K (rows past T read as zeros)
    auto issue_rows = [&](const uint16_t* tensor, int dst) {
        const int left = (T - row0) * (D * 2);
        const int nrec = left < BS * D * 2 ? left : BS * D * 2;
        const i32x4 rr = buffer_rsrc(tensor + head_off + (size_t)row0 * D, nrec);
#pragma unroll
        for (int n = 0; n < NDMA_R; ++n) {
            const int slot = n * 64 + lane;
            const int r = slot / DC, s = slot - (slot / DC) * DC;
            if (RSLOT % 64 == 0 || slot < RSLOT)
                dma16(lds0 + dst + n * 1024, r * (D * 2) + ((s ^ kswz<D>(r)) * 16), rr);
        }
    };

    // wait until at most n vector-memory operations (the ones just issued) are
    // outstanding; waiting for fewer is always safe, so take the largest constant <= n
    auto wait_le = [&](int n) {
        if (n >= 2 * NDMA + NDMA_R) {
            wait_vm<2 * NDMA + NDMA_R>();
        } else if (n >= NDMA + NDMA_R) {
            wait_vm<NDMA + NDMA_R>();
        } else if (n >= 2 * NDMA) {
            wait_vm<2 * NDMA>();
        } else if (n >= NDMA_R) {
            wait_vm<NDMA_R>();
        } else if (n >= NDMA) {
            wait_vm<NDMA>();
        } else {
            wait_vm<0>();
        }
    };

    // ---- prologue ---------------------------------------------------------------------
    float rho_r[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int row = row0 + qt * 32 + l32;
        rho_r[qt] = (RESHAPE && row < T) ? a.rho[(size_t)bh * T + row] : 0.f;
    }
    const int c0 = n_chunk > 0 ? chunk_base(0) : -1;
    int c1 = n_chunk > 1 ? chunk_base(1) : -1;
    issue(Kh, kdma, c0, k_off(0));
    issue_rows(a.q, v_off(0));
    issue(Kh, kdma, c1, k_off(1));
    if (c1 >= 0) {
        wait_vm<NDMA>();  // K(0) and the Q tile have landed; K(1) may be in flight
    } else {
        wait_vm<0>();
    }

    // Q^T operands from the Q tile: lane holds query l32 of tile qt, head dims
    // 16s + 8hi .. +7 (zero past D)
    bf16x8 qop[QT][DS];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int rl = qt * 32 + l32;
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            const int ch = 2 * s + hi;
            if (ch < DC) {
                qop[qt][s] = *(const lds_bf16x8*)(lds + v_off(0) + rl * ROWB + ((ch ^ kswz<D>(rl)) * 16));
            } else {
                qop[qt][s] = bf16x8{};
            }
        }
    }

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

    // S^T = K Q^T for the K chunk in stage `st`
    auto qk = [&](int st, f32x16 (&sc)[QT]) {
        const lds_u8* Ks = lds + k_off(st);
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
    // keys past T, or a chunk holding no key, score -inf
    auto mask = [&](int base, f32x16 (&sc)[QT]) {
        if (base >= 0 && base + 32 <= T) return;
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
            for (int x = 0; x < 16; ++x) {
                const int key = base + 8 * (x >> 2) + 4 * hi + (x & 3);
                if (base < 0 || key >= T) sc[qt][x] = -INFINITY;
            }
        }
    };
    // O^T += V^T P^T for the V chunk in stage `st`; the V^T operand is two
    // transpose reads of 4 rows each
    auto pv = [&](int st, const bf16x8 (&pp)[QT][2]) {
        const lds_u8* Vs = lds + v_off(st);
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
                    oacc[qt][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vv, pp[qt][ks], oacc[qt][dt], 0, 0, 0);
            }
        }
    };
    // probabilities of 4 scores against the running max: bf16 operand values and
    // their fp32 sum
    auto probs4 = [&](const f32x16& sc, int x0, float mc, bf16x8& pp, int y0) {
        float acc = 0.f;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[x0 + x], c2, -mc));
            acc += p;
            pp[y0 + x] = (__bf16)p;
        }
        return acc;
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
    // softmax of chunk scores `sc` against the running max; the rare case of a
    // probability reaching 2^64 rescales O and l and recomputes (all PV products
    // issued so far are in oacc by then)
    auto softmax_tail = [&](f32x16 (&sc)[QT], bf16x8 (&pp)[QT][2], float (&lsum)[QT], float (&mx)[QT]) {
        bool jump = false;
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) jump |= !(lsum[qt] < kJump);
        if (__builtin_amdgcn_ballot_w64(jump)) {
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
                if (!STATS) mx[qt] = chunk_max(sc[qt]);
                const float mnew = fmaxf(m_run[qt], mx[qt]);
                const float alpha = __builtin_amdgcn_exp2f((m_run[qt] - mnew) * c2);
                l_run[qt] *= alpha;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) oacc[qt][dt] *= alpha;
                m_run[qt] = mnew;
                const float mc = mnew * c2;
                lsum[qt] = probs4(sc[qt], 0, mc, pp[qt][0], 0) + probs4(sc[qt], 4, mc, pp[qt][0], 4) +
                           probs4(sc[qt], 8, mc, pp[qt][1], 0) + probs4(sc[qt], 12, mc, pp[qt][1], 4);
            }
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) l_run[qt] += lsum[qt];
    };

    // Software pipeline over chunks 0 .. n-1.  Step t issues the DMA of K(t+2) and
    // V(t) (into the stages K(t) and V(t-2) have left), then runs S(t+1) = K Q^T and
    // the P V product of chunk t-1 on the matrix cores, spread over the vector work
    // of chunk t's softmax.  The residual / output tile replaces the K stages once
    // the last K chunk has been read.
    f32x16 s_cur[QT];
    bf16x8 p_prev[QT][2];
    int r_issued = 0;
    if (n_chunk > 0) {
        qk(0, s_cur);
        mask(c0, s_cur);
    }
    // step 0: as the later steps, without a P V product yet
    {
        const int c2n = n_chunk > 2 ? chunk_base(2) : -1;
        issue(Kh, kdma, c2n, k_off(0));  // K(0) has been read
        issue(Vh, vdma, c0, v_off(0));   // the Q tile has been read
        int now = (c2n >= 0 ? NDMA : 0) + (c0 >= 0 ? NDMA : 0);
        if (RESHAPE && n_chunk <= 1) {  // no K chunk left to read
            issue_rows(a.resid, 0);
            r_issued = 1;
            now += NDMA_R;
        }
        wait_le(now);  // K(1)
        if (n_chunk > 0) {
            f32x16 s_nxt[QT];
            float lsum[QT], mx[QT];
            bf16x8 pp[QT][2];
            if (n_chunk > 1) qk(1, s_nxt);
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
                if (STATS) {
                    mx[qt] = chunk_max(s_cur[qt]);
                    m_top[qt] = fmaxf(m_top[qt], mx[qt]);
                }
                const float mc = m_run[qt] * c2;
                lsum[qt] = probs4(s_cur[qt], 0, mc, pp[qt][0], 0) + probs4(s_cur[qt], 4, mc, pp[qt][0], 4) +
                           probs4(s_cur[qt], 8, mc, pp[qt][1], 0) + probs4(s_cur[qt], 12, mc, pp[qt][1], 4);
            }
            softmax_tail(s_cur, pp, lsum, mx);
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
                p_prev[qt][0] = pp[qt][0];
                p_prev[qt][1] = pp[qt][1];
            }
            if (n_chunk > 1) {
#pragma unroll
                for (int qt = 0; qt < QT; ++qt) s_cur[qt] = s_nxt[qt];
                mask(c1, s_cur);
            }
        }
    }
    // rolling window of chunk bases: b_t = base(t), b_t1 = base(t+1)
    int b_t = n_chunk > 1 ? c1 : -1;
    int b_t1 = n_chunk > 2 ? chunk_base(2) : -1;
    for (int t = 1; t < n_chunk; ++t) {
        const int kst = t & 1;  // stage of K(t) and V(t)
        // refill: K(t+2) -> stage of K(t), V(t) -> stage of V(t-2); the residual
        // tile takes the K stages once the last K chunk (t) was read in step t-1
        const int cn2 = t + 2 < n_chunk ? chunk_base(t + 2) : -1;
        const int ct = b_t;
        issue(Kh, kdma, cn2, k_off(kst));
        issue(Vh, vdma, ct, v_off(kst));
        if (RESHAPE && t == n_chunk - 1) {
            issue_rows(a.resid, 0);
            r_issued = 1;
        }
        // K(t+1) and V(t-1) were issued one step earlier
        wait_le((cn2 >= 0 ? NDMA : 0) + (ct >= 0 ? NDMA : 0) + ((RESHAPE && t == n_chunk - 1) ? NDMA_R : 0));

        // interleaved block: S(t+1) and P V(t-1) on the matrix cores, softmax(t) on
        // the vector unit (after the last chunk the S product reads a stale stage
        // and is discarded)
        f32x16 s_nxt[QT];
        float lsum[QT], mx[QT];
        bf16x8 pp[QT][2];
        {
            const lds_u8* Ks = lds + k_off(kst ^ 1);
            const lds_u8* Vs = lds + v_off(kst ^ 1);
            bf16x8 kop[DS];
#pragma unroll
            for (int s = 0; s < DS; ++s) kop[s] = *(const lds_bf16x8*)(Ks + k_rd[s]);
            bf16x8 vop[DT][2];
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const bf16x4 v0 =
                        __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(Vs + v_rd[dt] + 16 * ks * ROWB));
                    const bf16x4 v1 =
                        __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(Vs + v_rd[dt] + (16 * ks + 8) * ROWB));
                    vop[dt][ks] = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
                }
            }
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
                s_nxt[qt] = f32x16{};
                lsum[qt] = 0.f;
            }
            if (STATS) {
#pragma unroll
                for (int qt = 0; qt < QT; ++qt) {
                    mx[qt] = chunk_max(s_cur[qt]);
                    m_top[qt] = fmaxf(m_top[qt], mx[qt]);
                }
            }
            // 4 S^T k-steps and 2 x 2 P V steps, each followed by one quarter of
            // the softmax's exponentials
#pragma unroll
            for (int k = 0; k < DS + 2 * DT; ++k) {
                __builtin_amdgcn_sched_barrier(0);
                if (k < DS) {
#pragma unroll
                    for (int qt = 0; qt < QT; ++qt)
                        s_nxt[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[k], qop[qt][k], s_nxt[qt], 0, 0, 0);
                } else {
                    const int dt = (k - DS) >> 1, ks = (k - DS) & 1;
#pragma unroll
                    for (int qt = 0; qt < QT; ++qt)
                        oacc[qt][dt] =
                            __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[dt][ks], p_prev[qt][ks], oacc[qt][dt], 0, 0, 0);
                }
                // softmax quarter(s): 4 x QT groups of 4 scores spread over the steps
                constexpr int NQ = 4 * QT;
                constexpr int NSTEP = DS + 2 * DT;
#pragma unroll
                for (int q = 0; q < NQ; ++q) {
                    if (q * NSTEP / NQ == k) {
                        const int qt = q / 4, part = q % 4;
                        lsum[qt] += probs4(s_cur[qt], 4 * part, m_run[qt] * c2, pp[qt][part >> 1], 4 * (part & 1));
                    }
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        softmax_tail(s_cur, pp, lsum, mx);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            p_prev[qt][0] = pp[qt][0];
            p_prev[qt][1] = pp[qt][1];
            s_cur[qt] = s_nxt[qt];
        }
        if (t + 1 < n_chunk) mask(b_t1, s_cur);
        b_t = b_t1;
        b_t1 = cn2;
    }
    if (RESHAPE && !r_issued) {  // a block with no kept key block
        issue_rows(a.resid, 0);
        r_issued = 1;
    }
    wait_vm<0>();
    if (n_chunk > 0) pv((n_chunk - 1) & 1, p_prev);  // P V of the last chunk

    // ---- epilogue: O = factor * acc (+ R) into the tile in LDS, then row stores -----
    lds_u8* const Ot = lds;  // residual / output tile over the K stages
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
