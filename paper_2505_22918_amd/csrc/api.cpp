// C ABI of librettention: host-side argument checks, then launches on the
// caller's stream.  Nothing here allocates device memory or synchronises.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <algorithm>
#include <initializer_list>
#include <numeric>
#include <utility>

#include "../../include/rettention.h"
#include "kernels.h"

namespace {

thread_local char g_err[512] = "";

rt_status fail(rt_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return s;
}

rt_status ok() {
    g_err[0] = '\0';
    return RT_OK;
}

rt_status hip_status(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(RT_EHIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Shape checks shared by every tensor call; sets *empty when there is no work.
rt_status check_dims(const rt_dims& d, bool* empty) {
    if (d.B < 0 || d.H < 0 || d.T < 0) return fail(RT_EINVAL, "negative dims B=%d H=%d T=%d", d.B, d.H, d.T);
    if (d.D != 64 && d.D != 72) return fail(RT_EUNSUPPORTED, "head width D=%d (supported: 64, 72)", d.D);
    const int64_t rows = (int64_t)d.B * d.H * d.T;
    if (rows * d.D >= (int64_t)1 << 40) return fail(RT_EINVAL, "tensor too large");
    if ((int64_t)d.B * d.H >= (int64_t)1 << 24) return fail(RT_EINVAL, "B*H too large");
    // buffer record counts and offsets within one head are 32-bit, with 2^30
    // kept free as the out-of-range offset that reads zeros
    if ((int64_t)d.T * d.D * 2 > (int64_t)1 << 30) return fail(RT_EINVAL, "T=%d too long for one head", d.T);
    *empty = rows == 0;
    return RT_OK;
}

rt_status check_tensor(const void* p, const char* name) {
    if (!p) return fail(RT_EINVAL, "%s is NULL", name);
    if (!aligned16(p)) return fail(RT_EINVAL, "%s is not 16-byte aligned", name);
    return RT_OK;
}

rt_status check_stat(const void* p, const char* name) {
    if (!p) return fail(RT_EINVAL, "%s is NULL", name);
    if ((reinterpret_cast<uintptr_t>(p) & 3u) != 0) return fail(RT_EINVAL, "%s is not 4-byte aligned", name);
    return RT_OK;
}

rt_status check_block(int32_t block) {
    if (block != 32 && block != 64) return fail(RT_EUNSUPPORTED, "block=%d (supported: 32, 64)", block);
    return RT_OK;
}

#define RT_TRY(expr)                  \
    do {                              \
        rt_status _s = (expr);        \
        if (_s != RT_OK) return _s;   \
    } while (0)

rt_status check_qkv(const void* q, const void* k, const void* v, void* o) {
    RT_TRY(check_tensor(q, "q"));
    RT_TRY(check_tensor(k, "k"));
    RT_TRY(check_tensor(v, "v"));
    RT_TRY(check_tensor(o, "o"));
    return RT_OK;
}

int64_t tensor_bytes(const rt_dims& d, int64_t elem) { return (int64_t)d.B * d.H * d.T * d.D * elem; }

// The byte ranges [a, a + na) and [b, b + nb) share a byte.
bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

// Attention outputs are written by one work item per query block while every
// work item reads K and V (and its own Q rows), so an output that overlaps an
// input would be read back by other work items; no overlap is accepted.
rt_status check_no_overlap(const void* out, int64_t out_bytes, const char* out_name,
                           std::initializer_list<std::pair<const void*, int64_t>> ins, const char* in_names) {
    for (const auto& in : ins)
        if (in.first && overlaps(out, out_bytes, in.first, in.second))
            return fail(RT_EINVAL, "%s overlaps %s (outputs must not alias the inputs)", out_name, in_names);
    return RT_OK;
}

// Optional row statistics: they must not overlap each other, o or the other
// listed buffers.
rt_status check_stats_overlap(const rt_dims& d, const float* row_max, const float* row_sum, const void* o,
                              std::initializer_list<std::pair<const void*, int64_t>> others) {
    const int64_t ns = tensor_bytes(d, 4) / d.D, nt = tensor_bytes(d, 2);
    for (const float* st : {row_max, row_sum}) {
        if (!st) continue;
        RT_TRY(check_no_overlap(st, ns, "row_max / row_sum", {{o, nt}}, "o"));
        RT_TRY(check_no_overlap(st, ns, "row_max / row_sum", others, "another output or input"));
    }
    if (row_max && row_sum && overlaps(row_max, ns, row_sum, ns))
        return fail(RT_EINVAL, "row_max overlaps row_sum");
    return RT_OK;
}

rt::AttnArgs base_args(const void* q, const void* k, const void* v, const rt_dims& d, int32_t block,
                       void* o, float* row_max, float* row_sum) {
    rt::AttnArgs a{};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.o = static_cast<uint16_t*>(o);
    a.row_max = row_max;
    a.row_sum = row_sum;
    a.T = d.T;
    a.n_blk = (int32_t)ceil_div(d.T, block);
    const int64_t items = (int64_t)d.B * d.H * a.n_blk;
    a.n_items = (int32_t)items;
    a.per_xcd = (int32_t)ceil_div(items, 8);
    a.scale_nat = (float)(1.0 / std::sqrt((double)d.D));
    a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d.D));
    return a;
}

rt_status check_items(const rt_dims& d, int32_t block) {
    const int64_t items = (int64_t)d.B * d.H * ceil_div(d.T, block);
    if (8 * ceil_div(items, 8) > INT32_MAX) return fail(RT_EINVAL, "too many query blocks");
    return RT_OK;
}

rt_status check_bsr(const rt_bsr* m, const rt_dims& d) {
    if (!m) return fail(RT_EINVAL, "mask is NULL");
    RT_TRY(check_block(m->block));
    const int64_t nb = ceil_div(d.T, m->block);
    if (m->n_qblk != nb) return fail(RT_EINVAL, "n_qblk=%d but ceil(T/block)=%lld", m->n_qblk, (long long)nb);
    if (m->nnz < 0) return fail(RT_EINVAL, "nnz=%d", m->nnz);
    if (nb > 0 && m->nnz == 0) return fail(RT_EINVAL, "empty mask: every query block needs a kept key block (Eq.5)");
    if (nb > 0 && (!m->row_ptr || !m->col_idx)) return fail(RT_EINVAL, "row_ptr / col_idx is NULL");
    const int64_t bh = (int64_t)d.B * d.H;
    if (m->n_masks != 0 && m->n_masks != 1 && m->n_masks != d.H && m->n_masks != bh)
        return fail(RT_EINVAL, "n_masks=%d (need 1, H=%d or B*H=%lld)", m->n_masks, d.H, (long long)bh);
    return RT_OK;
}

void set_mask(rt::AttnArgs& a, const rt_bsr* m, const rt_dims& d) {
    a.row_ptr = m->row_ptr;
    a.col_idx = m->col_idx;
    a.nnz = m->nnz;
    a.n_masks = m->n_masks > 1 ? m->n_masks : 1;
    a.heads = d.H;
}

int64_t lcm64(int64_t a, int64_t b) { return a / std::gcd(a, b) * b; }

// Validates a pattern and fills the launch arguments (mask and outputs aside).
rt_status pattern_args(const rt_pattern* p, int32_t T, int32_t block, rt::IndexArgs* out, int64_t* nnz) {
    if (!p) return fail(RT_EINVAL, "pattern is NULL");
    RT_TRY(check_block(block));
    if (T < 1) return fail(RT_EINVAL, "T=%d (need T >= 1)", T);
    const int64_t nb = ceil_div(T, block);
    if (nb > 4096) return fail(RT_EUNSUPPORTED, "ceil(T/block)=%lld exceeds 4096 blocks", (long long)nb);
    rt::IndexArgs a{};
    a.kind = p->kind;
    a.T = T;
    a.block = block;
    a.n_blk = (int32_t)nb;
    a.keep = p->keep;
    a.lcm = 1;
    if (p->n_masks < 0) return fail(RT_EINVAL, "n_masks=%d", p->n_masks);
    a.n_masks = p->n_masks > 1 ? p->n_masks : 1;
    if (a.n_masks > 1 && p->kind != RT_PAT_EXPLICIT)
        return fail(RT_EINVAL, "n_masks=%d: the window patterns are the same for every head", p->n_masks);
    if (a.n_masks > 1 && (int64_t)a.n_masks * nb > 32768)
        return fail(RT_EUNSUPPORTED, "n_masks * ceil(T/block) = %lld exceeds 32768",
                    (long long)a.n_masks * nb);
    switch (p->kind) {
        case RT_PAT_EXPLICIT:
            *nnz = -1;
            break;
        case RT_PAT_LOCAL2D: {
            if (p->grid_h < 1 || p->grid_w < 1 || p->grid_h > 65535 || p->grid_w > 65535)
                return fail(RT_EINVAL, "grid %dx%d out of range", p->grid_h, p->grid_w);
            if ((int64_t)p->grid_h * p->grid_w != T)
                return fail(RT_EINVAL, "grid_h*grid_w=%lld != T=%d", (long long)p->grid_h * p->grid_w, T);
            if (p->keep < 1) return fail(RT_EINVAL, "keep=%d (need >= 1)", p->keep);
            a.grid_h = p->grid_h;
            a.grid_w = p->grid_w;
            const int64_t last = T - (nb - 1) * block;
            a.lcm = nb > 1 ? lcm64(block, last) : last;
            *nnz = nb * std::min<int64_t>(p->keep, nb);
            break;
        }
        case RT_PAT_VIDEO3D: {
            if (p->grid_h < 1 || p->grid_w < 1 || p->frames < 1 || p->grid_h > 65535 || p->grid_w > 65535 ||
                p->frames > 65535 || p->n_text < 0)
                return fail(RT_EINVAL, "video grid %dx%dx%d / n_text=%d out of range", p->frames, p->grid_h,
                            p->grid_w, p->n_text);
            if ((int64_t)p->n_text + (int64_t)p->frames * p->grid_h * p->grid_w != T)
                return fail(RT_EINVAL, "n_text + frames*grid_h*grid_w != T=%d", T);
            if (p->keep < 1) return fail(RT_EINVAL, "keep=%d (need >= 1)", p->keep);
            a.grid_h = p->grid_h;
            a.grid_w = p->grid_w;
            a.frames = p->frames;
            a.n_text = p->n_text;
            const int64_t ntb = ceil_div(p->n_text, block);
            a.n_tblk = (int32_t)ntb;
            const int64_t nv = nb - ntb;
            if (nv >= 1) {
                const int64_t last = T - (nb - 1) * block;
                a.lcm = nv > 1 ? lcm64(block, last) : last;
            }
            *nnz = ntb * ntb + (nb - ntb) * (ntb + std::min<int64_t>(p->keep, nv));
            break;
        }
        default:
            return fail(RT_EINVAL, "unknown pattern kind %d", p->kind);
    }
    *out = a;
    return RT_OK;
}

}  // namespace

extern "C" {

const char* rt_status_str(rt_status s) {
    switch (s) {
        case RT_OK: return "ok";
        case RT_EINVAL: return "invalid argument";
        case RT_EUNSUPPORTED: return "unsupported configuration";
        case RT_ECAPACITY: return "output capacity too small";
        case RT_EHIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char* rt_last_error(void) { return g_err; }

int32_t rt_version(void) { return 100; }

rt_status rt_index_size(const rt_pattern* pattern, int32_t T, int32_t block, int32_t* nnz_out) {
    if (!nnz_out) return fail(RT_EINVAL, "nnz_out is NULL");
    rt::IndexArgs a{};
    int64_t nnz = 0;
    RT_TRY(pattern_args(pattern, T, block, &a, &nnz));
    if (pattern->kind == RT_PAT_EXPLICIT) {
        if (!pattern->host_mask) return fail(RT_EINVAL, "EXPLICIT pattern needs host_mask for sizing");
        nnz = 0;
        const int64_t rows = (int64_t)a.n_masks * a.n_blk;
        for (int64_t r = 0; r < rows; ++r) {
            const uint8_t* row = pattern->host_mask + r * a.n_blk;
            int64_t kept = 0;
            for (int64_t j = 0; j < a.n_blk; ++j) kept += row[j] != 0;
            // Eq.5 normalises over the kept keys: an empty kept set has no softmax
            if (kept == 0)
                return fail(RT_EINVAL, "mask %lld, query block %lld keeps no key block (Eq.5 needs one)",
                            (long long)(r / a.n_blk), (long long)(r % a.n_blk));
            nnz += kept;
        }
    }
    if (nnz > INT32_MAX) return fail(RT_EINVAL, "nnz exceeds int32");
    *nnz_out = (int32_t)nnz;
    return ok();
}

rt_status rt_index_build(const rt_pattern* pattern, int32_t T, int32_t block, int32_t* row_ptr,
                         int32_t* col_idx, int32_t capacity, void* stream) {
    rt::IndexArgs a{};
    int64_t nnz = 0;
    RT_TRY(pattern_args(pattern, T, block, &a, &nnz));
    if (!row_ptr || !col_idx) return fail(RT_EINVAL, "row_ptr / col_idx is NULL");
    if (capacity < 0) return fail(RT_EINVAL, "capacity=%d", capacity);
    if (pattern->kind == RT_PAT_EXPLICIT) {
        if (!pattern->mask) return fail(RT_EINVAL, "EXPLICIT pattern needs a device mask");
        if (pattern->host_mask) {
            int32_t need = 0;
            RT_TRY(rt_index_size(pattern, T, block, &need));
            nnz = need;
        }
    }
    if (nnz >= 0 && capacity < nnz)
        return fail(RT_ECAPACITY, "capacity=%d but the mask has %lld entries", capacity, (long long)nnz);
    a.mask = pattern->mask;
    a.row_ptr = row_ptr;
    a.col_idx = col_idx;
    a.capacity = capacity;
    return hip_status(rt::launch_index_build(a, static_cast<hipStream_t>(stream)), "index build launch");
}

rt_status rt_bsr_check(const rt_bsr* mask, const int32_t* host_row_ptr, const int32_t* host_col_idx) {
    if (!mask) return fail(RT_EINVAL, "mask is NULL");
    RT_TRY(check_block(mask->block));
    if (mask->n_qblk < 0 || mask->nnz < 0 || mask->n_masks < 0)
        return fail(RT_EINVAL, "n_qblk=%d nnz=%d n_masks=%d", mask->n_qblk, mask->nnz, mask->n_masks);
    const int64_t nb = mask->n_qblk, nm = mask->n_masks > 1 ? mask->n_masks : 1;
    if (nb == 0) return mask->nnz == 0 ? ok() : fail(RT_EINVAL, "nnz=%d for a mask without rows", mask->nnz);
    if (!host_row_ptr || !host_col_idx) return fail(RT_EINVAL, "host_row_ptr / host_col_idx is NULL");
    int64_t last = 0;
    for (int64_t m = 0; m < nm; ++m) {
        const int32_t* rp = host_row_ptr + m * (nb + 1);
        for (int64_t i = 0; i < nb; ++i) {
            if (rp[i] < 0 || rp[i + 1] > mask->nnz)
                return fail(RT_EINVAL, "mask %lld row %lld: offsets [%d, %d) outside [0, nnz=%d]", (long long)m,
                            (long long)i, rp[i], rp[i + 1], mask->nnz);
            // Eq.5 normalises over the kept keys: an empty kept set has no softmax
            if (rp[i + 1] <= rp[i])
                return fail(RT_EINVAL, "mask %lld, query block %lld keeps no key block (Eq.5 needs one)",
                            (long long)m, (long long)i);
            for (int32_t e = rp[i]; e < rp[i + 1]; ++e) {
                const int32_t c = host_col_idx[e];
                if (c < 0 || c >= nb)
                    return fail(RT_EINVAL, "mask %lld row %lld: key block %d outside [0, %lld)", (long long)m,
                                (long long)i, c, (long long)nb);
                if (e > rp[i] && c <= host_col_idx[e - 1])
                    return fail(RT_EINVAL, "mask %lld row %lld: key blocks not strictly ascending", (long long)m,
                                (long long)i);
            }
        }
        last = std::max<int64_t>(last, rp[nb]);
    }
    if (last != mask->nnz)
        return fail(RT_EINVAL, "nnz=%d but the row offsets end at %lld", mask->nnz, (long long)last);
    return ok();
}

namespace {

// Shape checks of the dynamic index build; fills the counts it needs.
rt_status dynamic_shape(const rt_dims& dims, int32_t block, int32_t keep, int64_t* n_blk, int64_t* kk,
                        int64_t* nnz, int64_t* ws_bytes) {
    bool empty = false;
    RT_TRY(check_dims(dims, &empty));
    RT_TRY(check_block(block));
    if (keep < 1) return fail(RT_EINVAL, "keep=%d (need >= 1)", keep);
    const int64_t nb = ceil_div(dims.T, block);
    if (nb > 4096) return fail(RT_EUNSUPPORTED, "ceil(T/block)=%lld exceeds 4096 blocks", (long long)nb);
    const int64_t bh = (int64_t)dims.B * dims.H;
    *n_blk = nb;
    *kk = std::min<int64_t>(keep, nb);
    *nnz = bh * nb * *kk;
    if (*nnz > INT32_MAX || bh * (nb + 1) > INT32_MAX) return fail(RT_EINVAL, "mask too large for int32 offsets");
    *ws_bytes = 2 * bh * nb * dims.D * (int64_t)sizeof(float);
    return RT_OK;
}

}  // namespace

rt_status rt_dynamic_index_workspace(rt_dims dims, int32_t block, int32_t keep, int64_t* bytes) {
    if (!bytes) return fail(RT_EINVAL, "bytes is NULL");
    int64_t nb, kk, nnz, ws;
    RT_TRY(dynamic_shape(dims, block, keep, &nb, &kk, &nnz, &ws));
    *bytes = ws;
    return ok();
}

rt_status rt_dynamic_index_noalloc(const void* q, const void* k, rt_dims dims, int32_t block, int32_t keep,
                                   int32_t* row_ptr, int32_t* col_idx, int32_t capacity, void* stream) {
    int64_t nb, kk, nnz, ws;
    RT_TRY(dynamic_shape(dims, block, keep, &nb, &kk, &nnz, &ws));
    if (ws > rt::kDynScratchFloats * (int64_t)sizeof(float))
        return fail(RT_ECAPACITY, "the shape needs %lld workspace bytes, the allocation-free build holds %lld",
                    (long long)ws, (long long)(rt::kDynScratchFloats * (int64_t)sizeof(float)));
    if ((int64_t)dims.B * dims.H * dims.T == 0) return ok();
    float* scratch = nullptr;
    RT_TRY(hip_status(rt::dynamic_scratch(&scratch), "workspace address"));
    return rt_dynamic_index(q, k, dims, block, keep, row_ptr, col_idx, capacity, scratch, ws, stream);
}

rt_status rt_dynamic_index(const void* q, const void* k, rt_dims dims, int32_t block, int32_t keep,
                           int32_t* row_ptr, int32_t* col_idx, int32_t capacity, void* workspace,
                           int64_t workspace_bytes, void* stream) {
    int64_t nb, kk, nnz, ws;
    RT_TRY(dynamic_shape(dims, block, keep, &nb, &kk, &nnz, &ws));
    if ((int64_t)dims.B * dims.H * dims.T == 0) return ok();
    RT_TRY(check_tensor(q, "q"));
    RT_TRY(check_tensor(k, "k"));
    RT_TRY(check_stat(row_ptr, "row_ptr"));
    RT_TRY(check_stat(col_idx, "col_idx"));
    RT_TRY(check_tensor(workspace, "workspace"));
    if (capacity < nnz)
        return fail(RT_ECAPACITY, "capacity=%d but the mask has %lld entries", capacity, (long long)nnz);
    if (workspace_bytes < ws)
        return fail(RT_ECAPACITY, "workspace of %lld bytes, %lld needed", (long long)workspace_bytes, (long long)ws);
    const int64_t nt = tensor_bytes(dims, 2);
    const int64_t nrp = (int64_t)dims.B * dims.H * (nb + 1) * 4, nci = nnz * 4;
    RT_TRY(check_no_overlap(row_ptr, nrp, "row_ptr", {{q, nt}, {k, nt}, {col_idx, nci}, {workspace, ws}},
                            "q, k, col_idx or the workspace"));
    RT_TRY(check_no_overlap(col_idx, nci, "col_idx", {{q, nt}, {k, nt}, {workspace, ws}}, "q, k or the workspace"));
    RT_TRY(check_no_overlap(workspace, ws, "workspace", {{q, nt}, {k, nt}}, "q or k"));
    rt::DynIndexArgs a{};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.B = dims.B;
    a.H = dims.H;
    a.T = dims.T;
    a.D = dims.D;
    a.block = block;
    a.n_blk = (int32_t)nb;
    a.keep = keep;
    a.qsum = static_cast<float*>(workspace);
    a.kmean = a.qsum + (size_t)dims.B * dims.H * nb * dims.D;
    a.row_ptr = row_ptr;
    a.col_idx = col_idx;
    return hip_status(rt::launch_dynamic_index(a, static_cast<hipStream_t>(stream)), "dynamic index launch");
}

rt_status rt_attn_full(const void* q, const void* k, const void* v, rt_dims dims, int32_t block, void* o,
                       float* row_max, float* row_sum, void* stream) {
    bool empty = false;
    RT_TRY(check_dims(dims, &empty));
    RT_TRY(check_block(block));
    if (empty) return ok();
    RT_TRY(check_qkv(q, k, v, o));
    if (row_max) RT_TRY(check_stat(row_max, "row_max"));
    if (row_sum) RT_TRY(check_stat(row_sum, "row_sum"));
    const int64_t nt = tensor_bytes(dims, 2);
    RT_TRY(check_no_overlap(o, nt, "o", {{q, nt}, {k, nt}, {v, nt}}, "q, k or v"));
    RT_TRY(check_stats_overlap(dims, row_max, row_sum, o, {}));
    RT_TRY(check_items(dims, block));
    rt::AttnArgs a = base_args(q, k, v, dims, block, o, row_max, row_sum);
    a.dense = 1;
    return hip_status(rt::launch_attention(a, dims.D, block, rt::kAttn, static_cast<hipStream_t>(stream)),
                      "full attention launch");
}

rt_status rt_attn_sparse(const void* q, const void* k, const void* v, rt_dims dims, const rt_bsr* mask,
                         void* o, float* row_max, float* row_sum, void* stream) {
    bool empty = false;
    RT_TRY(check_dims(dims, &empty));
    RT_TRY(check_bsr(mask, dims));
    if (empty) return ok();
    RT_TRY(check_qkv(q, k, v, o));
    if (row_max) RT_TRY(check_stat(row_max, "row_max"));
    if (row_sum) RT_TRY(check_stat(row_sum, "row_sum"));
    const int64_t nt = tensor_bytes(dims, 2);
    RT_TRY(check_no_overlap(o, nt, "o", {{q, nt}, {k, nt}, {v, nt}}, "q, k or v"));
    RT_TRY(check_stats_overlap(dims, row_max, row_sum, o, {}));
    RT_TRY(check_items(dims, mask->block));
    rt::AttnArgs a = base_args(q, k, v, dims, mask->block, o, row_max, row_sum);
    set_mask(a, mask, dims);
    return hip_status(rt::launch_attention(a, dims.D, mask->block, rt::kAttn, static_cast<hipStream_t>(stream)),
                      "sparse attention launch");
}

rt_status rt_attn_cache(const void* q, const void* k, const void* v, rt_dims dims, const rt_bsr* mask, void* o,
                        float* row_max, float* row_sum, float* rho, void* resid, void* stream) {
    bool empty = false;
    RT_TRY(check_dims(dims, &empty));
    RT_TRY(check_bsr(mask, dims));
    if (empty) return ok();
    RT_TRY(check_qkv(q, k, v, o));
    if (rho) RT_TRY(check_stat(rho, "rho"));
    RT_TRY(check_tensor(resid, "resid"));
    if (row_max) RT_TRY(check_stat(row_max, "row_max"));
    if (row_sum) RT_TRY(check_stat(row_sum, "row_sum"));
    const int64_t nt = tensor_bytes(dims, 2), ns = tensor_bytes(dims, 4) / dims.D;
    RT_TRY(check_no_overlap(o, nt, "o", {{q, nt}, {k, nt}, {v, nt}, {resid, nt}}, "q, k, v or resid"));
    RT_TRY(check_no_overlap(resid, nt, "resid", {{q, nt}, {k, nt}, {v, nt}}, "q, k or v"));
    if (rho)
        RT_TRY(check_no_overlap(rho, ns, "rho", {{q, nt}, {k, nt}, {v, nt}, {o, nt}, {resid, nt}},
                                "q, k, v, o or resid"));
    RT_TRY(check_stats_overlap(dims, row_max, row_sum, o, {{resid, nt}, {rho, ns}}));
    RT_TRY(check_items(dims, mask->block));
    rt::AttnArgs a = base_args(q, k, v, dims, mask->block, o, row_max, row_sum);
    set_mask(a, mask, dims);
    a.rho_out = rho;
    a.resid_out = static_cast<uint16_t*>(resid);
    return hip_status(rt::launch_attention(a, dims.D, mask->block, rt::kAttnCache, static_cast<hipStream_t>(stream)),
                      "caching-step launch");
}

rt_status rt_attn_postmask(const void* q, const void* k, const void* v, rt_dims dims, const rt_bsr* mask, void* o,
                           void* stream) {
    bool empty = false;
    RT_TRY(check_dims(dims, &empty));
    RT_TRY(check_bsr(mask, dims));
    if (empty) return ok();
    RT_TRY(check_qkv(q, k, v, o));
    const int64_t nt = tensor_bytes(dims, 2);
    RT_TRY(check_no_overlap(o, nt, "o", {{q, nt}, {k, nt}, {v, nt}}, "q, k or v"));
    RT_TRY(check_items(dims, mask->block));
    rt::AttnArgs a = base_args(q, k, v, dims, mask->block, o, nullptr, nullptr);
    set_mask(a, mask, dims);
    a.postmask = 1;
    return hip_status(rt::launch_attention(a, dims.D, mask->block, rt::kAttnCache, static_cast<hipStream_t>(stream)),
                      "post-softmax masking launch");
}

rt_status rt_cache_build(const void* o_full, const float* m_full, const float* l_full, const void* o_sparse,
                         const float* m_sparse, const float* l_sparse, rt_dims dims, float* rho, void* resid,
                         void* stream) {
    bool empty = false;
    RT_TRY(check_dims(dims, &empty));
    if (empty) return ok();
    RT_TRY(check_tensor(o_full, "o_full"));
    RT_TRY(check_tensor(o_sparse, "o_sparse"));
    RT_TRY(check_tensor(resid, "resid"));
    if (rho) {  // without a ratio the statistics are not read
        RT_TRY(check_stat(m_full, "m_full"));
        RT_TRY(check_stat(l_full, "l_full"));
        RT_TRY(check_stat(m_sparse, "m_sparse"));
        RT_TRY(check_stat(l_sparse, "l_sparse"));
        RT_TRY(check_stat(rho, "rho"));
    }
    {
        const int64_t nt = tensor_bytes(dims, 2), ns = tensor_bytes(dims, 4) / dims.D;
        const std::initializer_list<std::pair<const void*, int64_t>> ins = {
            {o_full, nt}, {o_sparse, nt}, {m_full, ns}, {l_full, ns}, {m_sparse, ns}, {l_sparse, ns}};
        RT_TRY(check_no_overlap(resid, nt, "resid", ins, "an input"));
        if (rho) {
            RT_TRY(check_no_overlap(rho, ns, "rho", ins, "an input"));
            RT_TRY(check_no_overlap(rho, ns, "rho", {{resid, nt}}, "resid"));
        }
    }
    const int64_t rows = (int64_t)dims.B * dims.H * dims.T;
    if (!rho) m_full = l_full = m_sparse = l_sparse = nullptr;
    return hip_status(rt::launch_cache_build(static_cast<const uint16_t*>(o_full), m_full, l_full,
                                             static_cast<const uint16_t*>(o_sparse), m_sparse, l_sparse, rows,
                                             dims.D, rho, static_cast<uint16_t*>(resid),
                                             static_cast<hipStream_t>(stream)),
                      "cache build launch");
}

rt_status rt_attn_sparse_reshape(const void* q, const void* k, const void* v, rt_dims dims, const rt_bsr* mask,
                                 const float* rho, const void* resid, float rho_delta, void* o, float* row_max,
                                 float* row_sum, void* stream) {
    bool empty = false;
    RT_TRY(check_dims(dims, &empty));
    RT_TRY(check_bsr(mask, dims));
    if (!std::isfinite(rho_delta)) return fail(RT_EINVAL, "rho_delta is not finite");
    if (empty) return ok();
    RT_TRY(check_qkv(q, k, v, o));
    if (rho) RT_TRY(check_stat(rho, "rho"));
    RT_TRY(check_tensor(resid, "resid"));
    if (row_max) RT_TRY(check_stat(row_max, "row_max"));
    if (row_sum) RT_TRY(check_stat(row_sum, "row_sum"));
    const int64_t nt = tensor_bytes(dims, 2), ns = tensor_bytes(dims, 4) / dims.D;
    RT_TRY(check_no_overlap(o, nt, "o", {{q, nt}, {k, nt}, {v, nt}, {resid, nt}, {rho, ns}},
                            "q, k, v, resid or rho"));
    RT_TRY(check_stats_overlap(dims, row_max, row_sum, o, {{resid, nt}, {rho, ns}}));
    RT_TRY(check_items(dims, mask->block));
    rt::AttnArgs a = base_args(q, k, v, dims, mask->block, o, row_max, row_sum);
    set_mask(a, mask, dims);
    a.rho = rho;
    a.resid = static_cast<const uint16_t*>(resid);
    a.rho_delta = rho_delta;
    return hip_status(rt::launch_attention(a, dims.D, mask->block, rt::kAttnReshape, static_cast<hipStream_t>(stream)),
                      "sparse+reshape launch");
}

rt_status rt_reshape_apply(const void* o_sparse, const float* rho, const void* resid, float rho_delta,
                           rt_dims dims, void* o, void* stream) {
    bool empty = false;
    RT_TRY(check_dims(dims, &empty));
    if (!std::isfinite(rho_delta)) return fail(RT_EINVAL, "rho_delta is not finite");
    if (empty) return ok();
    RT_TRY(check_tensor(o_sparse, "o_sparse"));
    RT_TRY(check_tensor(resid, "resid"));
    RT_TRY(check_tensor(o, "o"));
    if (rho) RT_TRY(check_stat(rho, "rho"));
    {
        const int64_t nt = tensor_bytes(dims, 2), ns = tensor_bytes(dims, 4) / dims.D;
        RT_TRY(check_no_overlap(o, nt, "o", {{o_sparse, nt}, {resid, nt}, {rho, ns}}, "o_sparse, resid or rho"));
    }
    const int64_t rows = (int64_t)dims.B * dims.H * dims.T;
    return hip_status(rt::launch_reshape_apply(static_cast<const uint16_t*>(o_sparse), rho,
                                               static_cast<const uint16_t*>(resid), rho_delta, rows, dims.D,
                                               static_cast<uint16_t*>(o), static_cast<hipStream_t>(stream)),
                      "reshape launch");
}

}  // extern "C"
