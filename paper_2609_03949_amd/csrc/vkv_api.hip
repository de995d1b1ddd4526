// vkv_api.hip -- the C ABI of libvkv: validation, workspace layout, launches.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "vkv_internal.h"

using namespace vkv;

constexpr int TIMING_SLOTS = 512;  // score launches timed between two vkv_score_timing calls

// The workspace of vkv_step_run_static: one per device, held until the process
// ends.  In host code `scratch` only names the symbol; its device address is
// taken once per device with hipGetSymbolAddress (in vkv_create) and used
// everywhere the host hands it to the kernels.
static __device__ __align__(256) uint8_t scratch[VKV_STATIC_WS_BYTES];

struct vkv_ctx {
    int device;
    int debug_rows;
    void* scratch_ptr;     // this device's address of `scratch`
    double* gram;          // [1024] device scratch for the contractivity check
    int timing;            // vkv_step_run records events around its score launch
    hipEvent_t* tev;       // [2 * TIMING_SLOTS] start/end events of timed score launches
    int tcount;            // timed launches recorded since the last read
    char err[512];
};

static thread_local char g_err[512];

static int fail(vkv_ctx* ctx, int code, const char* fmt, ...) {
    char* buf = ctx ? ctx->err : g_err;
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, 512, fmt, ap);
    va_end(ap);
    return code;
}

#define HIP_TRY(ctx, expr)                                                                 \
    do {                                                                                   \
        hipError_t _e = (expr);                                                            \
        if (_e != hipSuccess) return fail((ctx), VKV_E_HIP, "%s: %s", #expr, hipGetErrorString(_e)); \
    } while (0)

static inline bool al16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
static inline size_t up256(size_t v) { return (v + 255) & ~(size_t)255; }

// ------------------------------------------------------------ validation

static int index_width(const vkv_step* st) {
    return ((st->mode & 1) ? D_ROPE : 0) + ((st->mode & 2) ? st->r : 0);
}

static int check_step(vkv_ctx* ctx, const vkv_step* st) {
    if (!st) return fail(ctx, VKV_E_ARG, "step is NULL");
    if (st->B < 1 || st->B > 65535) return fail(ctx, VKV_E_SHAPE, "B=%lld outside [1, 65535]", (long long)st->B);
    if (st->H < 1 || st->H > 128) return fail(ctx, VKV_E_SHAPE, "H=%lld outside [1, 128]", (long long)st->H);
    if (st->T < 1 || st->T >= (1ll << 31)) return fail(ctx, VKV_E_SHAPE, "T=%lld outside [1, 2^31)", (long long)st->T);
    if (st->W < 0 || st->W > st->T) return fail(ctx, VKV_E_SHAPE, "W=%lld outside [0, T]", (long long)st->W);
    if (st->mode < 1 || st->mode > 3) return fail(ctx, VKV_E_ARG, "mode=%d is not a VKV_MODE_*", st->mode);
    if (st->mode == VKV_MODE_ROPE) {
        if (st->r != 0) return fail(ctx, VKV_E_ARG, "mode ROPE needs r = 0 (got %d)", st->r);
    } else {
        if (st->r < 32 || st->r > 512 || st->r % 32)
            return fail(ctx, VKV_E_UNSUPPORTED, "r=%d: need a multiple of 32 in [32, 512]", st->r);
    }
    const int n = index_width(st);
    if (n % 32 || n > D_ROW) return fail(ctx, VKV_E_UNSUPPORTED, "index width %d", n);
    if (!st->q_lat || !st->q_rope || !st->cache) return fail(ctx, VKV_E_ARG, "q_lat, q_rope and cache are required");
    if (!al16(st->q_lat) || !al16(st->q_rope) || !al16(st->cache))
        return fail(ctx, VKV_E_ALIGN, "q_lat, q_rope and cache must be 16-byte aligned");
    if (st->cache_row_stride < D_ROW || st->cache_row_stride % 8)
        return fail(ctx, VKV_E_ALIGN, "cache_row_stride=%lld: need >= 576 and a multiple of 8",
                    (long long)st->cache_row_stride);
    if (st->cache_batch_stride % 8 || (st->B > 1 && st->cache_batch_stride < st->T * st->cache_row_stride))
        return fail(ctx, VKV_E_ALIGN, "cache_batch_stride=%lld invalid", (long long)st->cache_batch_stride);
    if (st->index) {
        if (!al16(st->index)) return fail(ctx, VKV_E_ALIGN, "index must be 16-byte aligned");
        const int cols = (st->index_has_rope ? D_ROPE : 0) + ((st->mode & 2) ? st->r : 0);
        if (st->index_row_stride < cols || st->index_row_stride % 8)
            return fail(ctx, VKV_E_ALIGN, "index_row_stride=%lld: need >= %d and a multiple of 8",
                        (long long)st->index_row_stride, cols);
        if (st->index_batch_stride % 8 || (st->B > 1 && st->index_batch_stride < st->T * st->index_row_stride))
            return fail(ctx, VKV_E_ALIGN, "index_batch_stride=%lld invalid", (long long)st->index_batch_stride);
        if ((st->mode & 1) && !st->index_has_rope)
            return fail(ctx, VKV_E_UNSUPPORTED, "modes with the branch need an index built with_rope");
    } else if (st->mode != VKV_MODE_ROPE) {
        return fail(ctx, VKV_E_ARG, "modes with a digest need the index");
    }
    if ((st->mode & 2) && (!st->P || !al16(st->P))) return fail(ctx, VKV_E_ARG, "digest modes need a 16-byte aligned P");
    return VKV_OK;
}

// ----------------------------------------------------- workspace layout

// Attention splits: the k + W rows every step attends are cut into
// base_splits splits of rps rows, about one workgroup per CU over the batch
// (one fewer per sequence when rows may be admitted); the admitted rows'
// capacity (cap, a worst case that is mostly unused) gets splits of its own,
// the capacity spread over as many splits as there are workgroups per
// sequence but at least rps rows each and at most ATT_MAX_SPLIT_ROWS, taken
// in turn by a bounded number of workgroups.  Splits past a sequence's actual
// row count do no work and the combine reads only the splits that hold rows,
// so a large cap costs workspace, not time.
static void attend_split(const vkv_step* st, int64_t k, int64_t cap, int64_t* splits, int64_t* rps,
                         int64_t* base_splits, int64_t* rps_adm, int64_t* adm_blocks) {
    const int64_t nfix = k + st->W;
    const int64_t groups = st->B * ((st->H + ATT_HEADS - 1) / ATT_HEADS);
    const int64_t want = std::max<int64_t>(1, (256 + groups - 1) / groups);      // ~1 workgroup per CU
    auto rows_for = [&](int64_t n, int64_t lo, int64_t parts) {
        int64_t rows = (n + parts - 1) / parts;
        rows = std::max<int64_t>(rows, lo);
        rows = std::min<int64_t>(rows, ATT_MAX_SPLIT_ROWS);
        return (rows + ATT_CHUNK - 1) / ATT_CHUNK * ATT_CHUNK;
    };
    // with admitted rows, one of the ~1-per-CU workgroups is left for them, so
    // that a few admitted rows do not start a second round of workgroups
    const int64_t rows = rows_for(nfix, 128, cap > 0 ? std::max<int64_t>(1, want - 1) : want);
    const int64_t nb = std::max<int64_t>(1, (nfix + rows - 1) / rows);
    const int64_t rest = std::max<int64_t>(0, nfix + cap - nb * rows);   // positions past the base splits
    const int64_t ra = rows_for(cap, rows, want);
    const int64_t nadm = (rest + ra - 1) / ra;
    *rps = rows;
    *base_splits = nb;
    *rps_adm = ra;
    *splits = nb + nadm;
    // the admitted splits are taken in turn by up to 4 want workgroups: one
    // split each up to a capacity of about 4 splits per workgroup of the
    // batch (a full admission then runs as independent workgroups; measured:
    // taking two splits per workgroup made the near-total admission of the
    // 16-sequence, 32768-row workload 34% slower), beyond it a few splits each
    *adm_blocks = std::min<int64_t>(nadm, 4 * want);
}

static int64_t flag_stride(int64_t A) { return (std::max<int64_t>(A, 1) + 63) / 64 * 64; }

static WsLayout layout(const vkv_step* st, int64_t k, int64_t cap) {
    WsLayout L{};
    const int64_t B = st->B, H = st->H;
    L.A = st->T - st->W;
    L.n = index_width(st);
    L.nblk = std::max<int64_t>(1, (L.A + CB_KEYS - 1) / CB_KEYS);
    L.cap = cap;
    const int64_t Aw = std::max<int64_t>(L.A, 1);
    const int64_t Af = flag_stride(L.A);
    size_t o = 0;
    L.qt = o; o = up256(o + (size_t)(B * H * L.n * 2));
    L.hsc = o; o = up256(o + (size_t)(B * H * 16));
    L.seq = o; o = up256(o + (size_t)(B * SQ_WORDS * 4));
    L.kt = o; o = up256(o + (size_t)(B * Aw * 4));
    L.flags = o; o = up256(o + (size_t)(B * Af));
    L.flags2 = o; o = up256(o + (size_t)(B * Af));
    L.blk = o; o = up256(o + (size_t)(B * L.nblk * BLK_WORDS * 4));
    L.cand = o; o = up256(o + (size_t)(B * Aw * 4));
    L.candkey = o; o = up256(o + (size_t)(B * Aw * 4));
    L.amb = o; o = up256(o + (size_t)(B * Aw * 4));
    L.ambkey = o; o = up256(o + (size_t)(B * Aw * 8));
    L.rmx = o; o = up256(o + (size_t)(B * H * RM_MAX_SPLIT * 12));
    // everything above is independent of k and cap; the attention partials last
    attend_split(st, k, cap, &L.splits, &L.rows_per_split, &L.base_splits, &L.rows_per_adm, &L.adm_blocks);
    const int64_t HG = (H + ATT_HEADS - 1) / ATT_HEADS;   // partials padded to whole head groups
    L.part_o = o; o = up256(o + (size_t)(B * L.splits * HG * ATT_HEADS * D_LAT * 2));
    L.part_ml = o; o = up256(o + (size_t)(B * L.splits * H * 2 * 4));
    L.total = o;
    return L;
}

static int check_ws(vkv_ctx* ctx, const void* ws, size_t bytes, size_t need) {
    if (!ws) return fail(ctx, VKV_E_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)ws & 255u) != 0) return fail(ctx, VKV_E_ALIGN, "workspace must be 256-byte aligned");
    if (bytes < need) return fail(ctx, VKV_E_WORKSPACE, "workspace of %zu bytes, need %zu", bytes, need);
    return VKV_OK;
}

static void index_operand(const vkv_step* st, const uint16_t** x, int64_t* xs, int64_t* xbs) {
    if (st->mode == VKV_MODE_ROPE && !st->index) {
        *x = st->cache + D_LAT;
        *xs = st->cache_row_stride;
        *xbs = st->cache_batch_stride;
        return;
    }
    const int off = (st->mode == VKV_MODE_DIGEST && st->index_has_rope) ? D_ROPE : 0;
    *x = st->index + off;
    *xs = st->index_row_stride;
    *xbs = st->index_batch_stride;
}

// A run of sequences [b0, b0 + nb) of a step: every per-sequence array (inputs,
// outputs and the workspace's, all with the sequence as leading dimension) is
// offset to b0 and the kernels see nb sequences.
struct Chunk {
    int64_t b0, nb;
};

// bytes per sequence of each workspace array (the leading-dimension strides of layout())
struct WsStrides {
    size_t qt, hsc, seq, kt, flags, blk, cand, amb, ambkey, part_o, part_ml;
};

static WsStrides ws_strides(const vkv_step* st, const WsLayout& L) {
    const int64_t H = st->H, Aw = std::max<int64_t>(L.A, 1);
    return WsStrides{(size_t)(H * L.n * 2), (size_t)(H * 16),
                     (size_t)(SQ_WORDS * 4), (size_t)(Aw * 4), (size_t)flag_stride(L.A),
                     (size_t)(L.nblk * BLK_WORDS * 4), (size_t)(Aw * 4), (size_t)(Aw * 4), (size_t)(Aw * 8),
                     (size_t)(L.splits * ((H + ATT_HEADS - 1) / ATT_HEADS) * ATT_HEADS * D_LAT * 2),
                     (size_t)(L.splits * H * 2 * 4)};
}

static QprepArgs qprep_args(const vkv_step* st, const WsLayout& L, char* w, Chunk c) {
    const WsStrides z = ws_strides(st, L);
    const int64_t b0 = c.b0;
    return QprepArgs{st->q_lat + b0 * st->H * D_LAT, st->q_rope + b0 * st->H * D_ROPE, st->P, (int)c.nb, (int)st->H,
                     st->r, st->mode, (int)L.n, reinterpret_cast<uint16_t*>(w + L.qt + b0 * z.qt),
                     reinterpret_cast<float*>(w + L.hsc + b0 * z.hsc), reinterpret_cast<uint32_t*>(w + L.seq + b0 * z.seq)};
}

static ScoreArgs score_args(const vkv_step* st, const WsLayout& L, char* w, Chunk c, float* key, float* ub,
                            float cert_mult) {
    const WsStrides z = ws_strides(st, L);
    const int64_t b0 = c.b0;
    ScoreArgs a{};
    index_operand(st, &a.x, &a.xs, &a.xbs);
    a.x += b0 * a.xbs;
    a.qt = reinterpret_cast<const uint16_t*>(w + L.qt + b0 * z.qt);
    a.hsc = reinterpret_cast<const float*>(w + L.hsc + b0 * z.hsc);
    a.eta = st->eta ? st->eta + b0 * st->T : nullptr;
    a.eps = st->eps ? st->eps + b0 * st->T : nullptr;
    a.gam = st->gam ? st->gam + b0 * st->T : nullptr;
    a.T = st->T;
    a.key = key ? key + b0 * L.A : nullptr;
    a.ub = ub ? ub + b0 * L.A : nullptr;
    a.kt = reinterpret_cast<float*>(w + L.kt + b0 * z.kt);
    a.seq = reinterpret_cast<uint32_t*>(w + L.seq + b0 * z.seq);
    a.A = L.A;
    a.B = (int)c.nb;
    a.H = (int)st->H;
    a.n = (int)L.n;
    a.cert_mult = cert_mult;
    return a;
}

static SelectArgs select_args(const vkv_step* st, const WsLayout& L, char* w, Chunk c) {
    const WsStrides z = ws_strides(st, L);
    const int64_t b0 = c.b0;
    SelectArgs a{};
    index_operand(st, &a.x, &a.xs, &a.xbs);
    a.x += b0 * a.xbs;
    a.qt = reinterpret_cast<const uint16_t*>(w + L.qt + b0 * z.qt);
    a.hsc = reinterpret_cast<const float*>(w + L.hsc + b0 * z.hsc);
    a.eta = st->eta ? st->eta + b0 * st->T : nullptr;
    a.eps = st->eps ? st->eps + b0 * st->T : nullptr;
    a.gam = st->gam ? st->gam + b0 * st->T : nullptr;
    a.T = st->T;
    a.seq = reinterpret_cast<uint32_t*>(w + L.seq + b0 * z.seq);
    a.kt = reinterpret_cast<const float*>(w + L.kt + b0 * z.kt);
    a.flags = reinterpret_cast<uint8_t*>(w + L.flags + b0 * z.flags);
    a.flags2 = reinterpret_cast<uint8_t*>(w + L.flags2 + b0 * z.flags);
    a.blk = reinterpret_cast<uint32_t*>(w + L.blk + b0 * z.blk);
    a.cand = reinterpret_cast<int32_t*>(w + L.cand + b0 * z.cand);
    a.candkey = reinterpret_cast<float*>(w + L.candkey + b0 * z.cand);
    a.amb = reinterpret_cast<int32_t*>(w + L.amb + b0 * z.amb);
    a.ambkey = reinterpret_cast<uint64_t*>(w + L.ambkey + b0 * z.ambkey);
    a.A = L.A;
    a.nblk = L.nblk;
    a.fstride = (int64_t)z.flags;
    a.B = (int)c.nb;
    a.H = (int)st->H;
    a.n = (int)L.n;
    a.cert_mult = 1.0f;
    return a;
}

static AttendArgs attend_args(const vkv_step* st, const WsLayout& L, char* w, Chunk c, int64_t k, const int32_t* sel,
                              const int32_t* adm, const int32_t* adm_count, int64_t cap, float scale, uint16_t* out,
                              float* lse) {
    const WsStrides z = ws_strides(st, L);
    const int64_t b0 = c.b0;
    AttendArgs a{};
    a.q_lat = st->q_lat + b0 * st->H * D_LAT;
    a.q_rope = st->q_rope + b0 * st->H * D_ROPE;
    a.cache = st->cache + b0 * st->cache_batch_stride;
    a.cs = st->cache_row_stride;
    a.cbs = st->cache_batch_stride;
    a.sel = sel ? sel + b0 * k : nullptr;
    a.adm = adm ? adm + b0 * cap : nullptr;
    a.adm_count = adm_count ? adm_count + b0 : nullptr;
    a.k = k;
    a.W = st->W;
    a.A = L.A;
    a.cap = cap;
    a.rows_per_split = L.rows_per_split;
    a.rows_per_adm = L.rows_per_adm;
    a.splits = (int)L.splits;
    a.base_splits = (int)L.base_splits;
    a.adm_blocks = (int)L.adm_blocks;
    a.B = (int)c.nb;
    a.H = (int)st->H;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.part_o = reinterpret_cast<uint16_t*>(w + L.part_o + b0 * z.part_o);
    a.part_ml = reinterpret_cast<float*>(w + L.part_ml + b0 * z.part_ml);
    a.out = out + b0 * st->H * D_LAT;
    a.lse = lse + b0 * st->H;
    return a;
}

// ------------------------------------------------------- debug row sets

static int debug_check_sel(vkv_ctx* ctx, const vkv_step* st, int64_t k, const int32_t* sel, hipStream_t s) {
    if (!ctx->debug_rows || k == 0) return VKV_OK;
    const int64_t A = st->T - st->W;
    std::vector<int32_t> h((size_t)(st->B * k));
    HIP_TRY(ctx, hipMemcpyAsync(h.data(), sel, h.size() * 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(ctx, hipStreamSynchronize(s));
    for (int64_t b = 0; b < st->B; ++b)
        for (int64_t i = 0; i < k; ++i) {
            const int32_t u = h[(size_t)(b * k + i)];
            if (u < 0 || u >= A) return fail(ctx, VKV_E_DEBUG_ROWS, "sel[%lld][%lld]=%d outside the archive", (long long)b, (long long)i, u);
            if (i > 0 && u <= h[(size_t)(b * k + i - 1)])
                return fail(ctx, VKV_E_DEBUG_ROWS, "sel[%lld] not strictly ascending at %lld", (long long)b, (long long)i);
        }
    return VKV_OK;
}

static int debug_check_adm(vkv_ctx* ctx, const vkv_step* st, int64_t k, const int32_t* sel, const int32_t* adm,
                           const int32_t* cnt, int64_t cap, hipStream_t s) {
    if (!ctx->debug_rows) return VKV_OK;
    const int64_t A = st->T - st->W;
    std::vector<int32_t> hs((size_t)(st->B * std::max<int64_t>(k, 1)));
    std::vector<int32_t> ha((size_t)(st->B * std::max<int64_t>(cap, 1)));
    std::vector<int32_t> hc((size_t)st->B);
    if (k) HIP_TRY(ctx, hipMemcpyAsync(hs.data(), sel, (size_t)(st->B * k) * 4, hipMemcpyDeviceToHost, s));
    if (cap) HIP_TRY(ctx, hipMemcpyAsync(ha.data(), adm, (size_t)(st->B * cap) * 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(ctx, hipMemcpyAsync(hc.data(), cnt, (size_t)st->B * 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(ctx, hipStreamSynchronize(s));
    for (int64_t b = 0; b < st->B; ++b) {
        const int64_t m = std::min<int64_t>(hc[(size_t)b], cap);
        if (hc[(size_t)b] < 0 || hc[(size_t)b] > A - k)
            return fail(ctx, VKV_E_DEBUG_ROWS, "adm_count[%lld]=%d impossible", (long long)b, hc[(size_t)b]);
        const int32_t* sb = hs.data() + b * k;
        for (int64_t i = 0; i < m; ++i) {
            const int32_t u = ha[(size_t)(b * cap + i)];
            if (u < 0 || u >= A) return fail(ctx, VKV_E_DEBUG_ROWS, "adm[%lld][%lld]=%d outside the archive", (long long)b, (long long)i, u);
            if (i > 0 && u <= ha[(size_t)(b * cap + i - 1)])
                return fail(ctx, VKV_E_DEBUG_ROWS, "adm[%lld] not strictly ascending", (long long)b);
            if (std::binary_search(sb, sb + k, u))
                return fail(ctx, VKV_E_DEBUG_ROWS, "adm[%lld] row %d is also selected", (long long)b, u);
        }
    }
    return VKV_OK;
}

// ================================================================ C ABI

extern "C" {

int vkv_version(void) { return 100; }

const char* vkv_status_string(int status) {
    switch (status) {
        case VKV_OK: return "ok";
        case VKV_E_ARG: return "invalid argument";
        case VKV_E_SHAPE: return "unsupported shape";
        case VKV_E_ALIGN: return "misaligned pointer or stride";
        case VKV_E_UNSUPPORTED: return "unsupported configuration";
        case VKV_E_NOT_CONTRACTIVE: return "digest basis not certified contractive";
        case VKV_E_HIP: return "HIP runtime error";
        case VKV_E_WORKSPACE: return "workspace missing or too small";
        case VKV_E_DEBUG_ROWS: return "row-set assertion failed";
        default: return "unknown status";
    }
}

const char* vkv_last_error(const vkv_ctx* ctx) { return ctx ? ctx->err : g_err; }

int vkv_create(vkv_ctx** out, int device) {
    if (!out) return fail(nullptr, VKV_E_ARG, "out is NULL");
    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess) return fail(nullptr, VKV_E_HIP, "hipGetDeviceCount: %s", hipGetErrorString(e));
    if (device < 0 || device >= ndev) return fail(nullptr, VKV_E_ARG, "device %d of %d", device, ndev);
    e = hipSetDevice(device);
    if (e != hipSuccess) return fail(nullptr, VKV_E_HIP, "hipSetDevice: %s", hipGetErrorString(e));
    vkv_ctx* c = (vkv_ctx*)calloc(1, sizeof(vkv_ctx));
    if (!c) return fail(nullptr, VKV_E_ARG, "out of host memory");
    c->device = device;
    e = hipGetSymbolAddress(&c->scratch_ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !c->scratch_ptr) {
        free(c);
        return fail(nullptr, VKV_E_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    }
    const char* dbg = getenv("VKV_DEBUG_ROWS");
    c->debug_rows = (dbg && dbg[0] && strcmp(dbg, "0") != 0) ? 1 : 0;
    e = hipMalloc(&c->gram, 1024 * sizeof(double));
    if (e != hipSuccess) {
        free(c);
        return fail(nullptr, VKV_E_HIP, "hipMalloc: %s", hipGetErrorString(e));
    }
    *out = c;
    return VKV_OK;
}

int vkv_destroy(vkv_ctx* ctx) {
    if (!ctx) return VKV_OK;
    (void)hipSetDevice(ctx->device);
    if (ctx->tev) {
        for (int i = 0; i < 2 * TIMING_SLOTS; ++i) (void)hipEventDestroy(ctx->tev[i]);
        free(ctx->tev);
    }
    (void)hipFree(ctx->gram);
    free(ctx);
    return VKV_OK;
}

int vkv_digest_build(vkv_ctx* ctx, const uint16_t* cache, int64_t B, int64_t T, int64_t cache_row_stride,
                     int64_t cache_batch_stride, const uint16_t* P, int32_t r, int32_t with_rope, uint16_t* index,
                     int64_t index_row_stride, int64_t index_batch_stride, float* eta, float* eps, float* gam,
                     void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    hipStream_t s = (hipStream_t)stream;
    if (!cache) return fail(ctx, VKV_E_ARG, "cache is NULL");
    if (B < 1 || B > 65535 || T < 1 || T >= (1ll << 31)) return fail(ctx, VKV_E_SHAPE, "B=%lld T=%lld", (long long)B, (long long)T);
    if (r < 0 || r > 512 || (r % 32)) return fail(ctx, VKV_E_UNSUPPORTED, "r=%d: need 0 or a multiple of 32 up to 512", r);
    if (r > 0 && (!P || !al16(P))) return fail(ctx, VKV_E_ARG, "P must be a 16-byte aligned device pointer");
    if (!al16(cache) || cache_row_stride < D_ROW || cache_row_stride % 8 || cache_batch_stride % 8 ||
        (B > 1 && cache_batch_stride < T * cache_row_stride))
        return fail(ctx, VKV_E_ALIGN, "cache strides");
    const int cols = (with_rope ? D_ROPE : 0) + r;
    if (index) {
        if (!al16(index) || index_row_stride < cols || index_row_stride % 8 || index_batch_stride % 8 ||
            (B > 1 && index_batch_stride < T * index_row_stride))
            return fail(ctx, VKV_E_ALIGN, "index strides");
    }
    const bool cert = eta != nullptr;
    if (cert && (!eps || !gam)) return fail(ctx, VKV_E_ARG, "eta, eps and gam go together");
    if (!cert && !index) return fail(ctx, VKV_E_ARG, "nothing to build");
    if (cert && r > 0) {
        // Gershgorin: ||P||_2^2 = lambda_max(P P^T) <= max_j sum_k |(P P^T)_jk|.  A row
        // passes if its sum was computed exactly and is <= 1, or if it is <= 1 - 2^-30
        // (a margin far above the fp64 rounding of the sum).
        HIP_TRY(ctx, launch_gram_rows(P, r, ctx->gram, s));
        std::vector<double> rows((size_t)1024);
        HIP_TRY(ctx, hipMemcpyAsync(rows.data(), ctx->gram, 1024 * 8, hipMemcpyDeviceToHost, s));
        HIP_TRY(ctx, hipStreamSynchronize(s));
        for (int j = 0; j < r; ++j) {
            const double g = rows[(size_t)j];
            const bool exact = rows[(size_t)(512 + j)] == 0.0;
            if (!((exact && g <= 1.0) || g <= 1.0 - 0x1p-30))
                return fail(ctx, VKV_E_NOT_CONTRACTIVE,
                            "Gershgorin bound of ||P||_2^2 is %.9g (row %d) > 1", g, j);
        }
    }
    DigestArgs a{cache, cache_row_stride, cache_batch_stride, P, r, with_rope ? 1 : 0, index,
                 index_row_stride, index_batch_stride, eta, eps, gam, B, T};
    HIP_TRY(ctx, launch_digest(a, s));
    return VKV_OK;
}

int vkv_workspace_size(const vkv_step* st, int64_t k, int64_t cap, size_t* bytes) {
    if (!bytes) return fail(nullptr, VKV_E_ARG, "bytes is NULL");
    int rc = check_step(nullptr, st);
    if (rc) return rc;
    const int64_t A = st->T - st->W;
    if (k < 0 || k > A) return fail(nullptr, VKV_E_ARG, "k=%lld outside [0, A=%lld]", (long long)k, (long long)A);
    if (cap < 0 || cap > A) return fail(nullptr, VKV_E_ARG, "cap=%lld outside [0, A]", (long long)cap);
    *bytes = layout(st, k, cap).total;
    return VKV_OK;
}

}  // extern "C"

// ------------------------------------------- validation and launch, per stage

static int check_prep(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes) {
    int rc = check_step(ctx, st);
    if (rc) return rc;
    return check_ws(ctx, ws, ws_bytes, layout(st, 0, 0).part_o);
}

static int check_cert_mult(vkv_ctx* ctx, float cert_mult) {
    if (!(cert_mult >= 0.f) || !(cert_mult < 1e30f))
        return fail(ctx, VKV_E_ARG, "cert_mult must be finite and >= 0 (1 = the sound bound)");
    return VKV_OK;
}

static int check_score(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, float* ub, float cert_mult) {
    int rc = check_prep(ctx, st, ws, ws_bytes);
    if (rc) return rc;
    if (ub && (rc = check_cert_mult(ctx, cert_mult))) return rc;
    if (ub && (!st->eta || !st->eps || !st->gam)) return fail(ctx, VKV_E_ARG, "ub needs eta, eps and gam");
    if (ub && st->mode == VKV_MODE_DIGEST) return fail(ctx, VKV_E_UNSUPPORTED, "the bound needs the branch summand in the key");
    return VKV_OK;
}

static int check_select(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, int32_t* sel,
                        double* theta) {
    int rc = check_prep(ctx, st, ws, ws_bytes);
    if (rc) return rc;
    const int64_t A = st->T - st->W;
    if (k < 0 || k > A) return fail(ctx, VKV_E_ARG, "k=%lld outside [0, A=%lld]", (long long)k, (long long)A);
    if (!theta || (k > 0 && !sel)) return fail(ctx, VKV_E_ARG, "sel and theta are required");
    return VKV_OK;
}

static int check_admit(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, const int32_t* sel,
                       const double* theta, const float* ub, float cert_mult, int32_t* adm, int32_t* adm_count,
                       int64_t cap) {
    int rc = check_prep(ctx, st, ws, ws_bytes);
    if (rc) return rc;
    if ((rc = check_cert_mult(ctx, cert_mult))) return rc;
    const int64_t A = st->T - st->W;
    if (st->mode == VKV_MODE_DIGEST) return fail(ctx, VKV_E_UNSUPPORTED, "admission needs the branch summand in the key");
    if (!st->eta || !st->eps || !st->gam) return fail(ctx, VKV_E_ARG, "admission needs eta, eps and gam");
    if (k < 0 || k > A) return fail(ctx, VKV_E_ARG, "k=%lld outside [0, A]", (long long)k);
    if (cap < 0 || cap > A) return fail(ctx, VKV_E_ARG, "cap=%lld outside [0, A]", (long long)cap);
    if (!theta || !adm_count || (A > 0 && !ub) || (cap > 0 && !adm) || (k > 0 && !sel))
        return fail(ctx, VKV_E_ARG, "sel, theta, ub, adm and adm_count are required");
    return VKV_OK;
}

static int check_attend(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, const int32_t* sel,
                        const int32_t* adm, const int32_t* adm_count, int64_t cap, float scale, uint16_t* out,
                        float* lse) {
    int rc = check_step(ctx, st);
    if (rc) return rc;
    const int64_t A = st->T - st->W;
    if (k < 0 || k > A) return fail(ctx, VKV_E_ARG, "k=%lld outside [0, A]", (long long)k);
    if (cap < 0 || cap > A) return fail(ctx, VKV_E_ARG, "cap=%lld outside [0, A]", (long long)cap);
    if (cap > 0 && (!adm || !adm_count)) return fail(ctx, VKV_E_ARG, "cap > 0 needs adm and adm_count");
    if (!out || !lse || (k > 0 && !sel)) return fail(ctx, VKV_E_ARG, "sel, out and lse are required");
    if (!al16(out)) return fail(ctx, VKV_E_ALIGN, "out must be 16-byte aligned");
    if (!(scale > 0.f) || !(scale < 1e30f)) return fail(ctx, VKV_E_ARG, "scale must be positive and finite");
    return check_ws(ctx, ws, ws_bytes, layout(st, k, cap).total);
}

static hipError_t run_prep(const vkv_step* st, char* w, Chunk c, hipStream_t s) {
    return launch_qprep(qprep_args(st, layout(st, 0, 0), w, c), s);
}

static hipError_t run_score(const vkv_step* st, char* w, Chunk c, float* key, float* ub, float cert_mult,
                            hipStream_t s, const double* thr = nullptr, bool no_keys = false) {
    ScoreArgs a = score_args(st, layout(st, 0, 0), w, c, key, ub, cert_mult);
    a.thr = thr ? thr + c.b0 * st->H : nullptr;
    a.no_keys = (no_keys && ub && !key) ? 1 : 0;
    return launch_score(a, s);
}

static hipError_t run_select(const vkv_step* st, char* w, Chunk c, int64_t k, int32_t* sel, double* theta,
                             hipStream_t s) {
    SelectArgs a = select_args(st, layout(st, 0, 0), w, c);
    a.sel = sel ? sel + c.b0 * k : nullptr;
    a.theta = theta + c.b0;
    a.k = k;
    return launch_select(a, s);
}

static hipError_t run_admit(const vkv_step* st, char* w, Chunk c, int64_t k, const int32_t* sel, const double* theta,
                            const float* ub, float cert_mult, int32_t* adm, int32_t* adm_count, int64_t cap,
                            hipStream_t s) {
    const WsLayout L = layout(st, 0, 0);
    SelectArgs a = select_args(st, L, w, c);
    a.cert_mult = cert_mult;
    a.ub = ub ? ub + c.b0 * L.A : nullptr;
    a.sel = sel ? const_cast<int32_t*>(sel) + c.b0 * k : nullptr;
    a.theta = const_cast<double*>(theta) + c.b0;
    a.adm = adm ? adm + c.b0 * cap : nullptr;
    a.adm_count = adm_count + c.b0;
    a.k = k;
    a.cap = cap;
    return launch_admit(a, s);
}

static hipError_t run_attend(const vkv_step* st, char* w, Chunk c, int64_t k, const int32_t* sel, const int32_t* adm,
                             const int32_t* adm_count, int64_t cap, float scale, uint16_t* out, float* lse,
                             hipStream_t s) {
    if (cap == 0) {
        adm = nullptr;
        adm_count = nullptr;
    }
    return launch_attend(attend_args(st, layout(st, k, cap), w, c, k, sel, adm, adm_count, cap, scale, out, lse), s);
}

static int ensure_timing_events(vkv_ctx* ctx) {
    if (ctx->tev) return VKV_OK;
    hipEvent_t* ev = (hipEvent_t*)calloc(2 * TIMING_SLOTS, sizeof(hipEvent_t));
    if (!ev) return fail(ctx, VKV_E_ARG, "out of host memory");
    for (int i = 0; i < 2 * TIMING_SLOTS; ++i) {
        hipError_t e = hipEventCreate(&ev[i]);
        if (e != hipSuccess) {
            for (int j = 0; j < i; ++j) (void)hipEventDestroy(ev[j]);
            free(ev);
            return fail(ctx, VKV_E_HIP, "hipEventCreate: %s", hipGetErrorString(e));
        }
    }
    ctx->tev = ev;
    return VKV_OK;
}

extern "C" {

int vkv_query_prep(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_prep(ctx, st, ws, ws_bytes);
    if (rc) return rc;
    HIP_TRY(ctx, run_prep(st, (char*)ws, Chunk{0, st->B}, (hipStream_t)stream));
    return VKV_OK;
}

int vkv_score(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, float* key, float* ub, float cert_mult,
              void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_score(ctx, st, ws, ws_bytes, ub, cert_mult);
    if (rc) return rc;
    HIP_TRY(ctx, run_score(st, (char*)ws, Chunk{0, st->B}, key, ub, cert_mult, (hipStream_t)stream));
    return VKV_OK;
}

int vkv_select(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, int32_t* sel, double* theta,
               void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_select(ctx, st, ws, ws_bytes, k, sel, theta);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(ctx, run_select(st, (char*)ws, Chunk{0, st->B}, k, sel, theta, s));
    return debug_check_sel(ctx, st, k, sel, s);
}

int vkv_admit(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, const int32_t* sel,
              const double* theta, const float* ub, float cert_mult, int32_t* adm, int32_t* adm_count, int64_t cap,
              void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_admit(ctx, st, ws, ws_bytes, k, sel, theta, ub, cert_mult, adm, adm_count, cap);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(ctx, run_admit(st, (char*)ws, Chunk{0, st->B}, k, sel, theta, ub, cert_mult, adm, adm_count, cap, s));
    return debug_check_adm(ctx, st, k, sel, adm, adm_count, cap, s);
}

int vkv_attend(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, const int32_t* sel,
               const int32_t* adm, const int32_t* adm_count, int64_t cap, float scale, uint16_t* out, float* lse,
               void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_attend(ctx, st, ws, ws_bytes, k, sel, adm, adm_count, cap, scale, out, lse);
    if (rc) return rc;
    HIP_TRY(ctx, run_attend(st, (char*)ws, Chunk{0, st->B}, k, sel, adm, adm_count, cap, scale, out, lse,
                            (hipStream_t)stream));
    return VKV_OK;
}

int vkv_set_timing(vkv_ctx* ctx, int enable) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    if (enable) {
        int rc = ensure_timing_events(ctx);
        if (rc) return rc;
    }
    ctx->timing = enable ? 1 : 0;
    ctx->tcount = 0;
    return VKV_OK;
}

int vkv_score_timing(vkv_ctx* ctx, float* ms, int max) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    if (!ms || max < 1) return fail(ctx, VKV_E_ARG, "ms and max >= 1 are required");
    const int n = std::min(ctx->tcount, max);
    for (int i = 0; i < n; ++i) {
        HIP_TRY(ctx, hipEventSynchronize(ctx->tev[2 * i + 1]));
        HIP_TRY(ctx, hipEventElapsedTime(&ms[i], ctx->tev[2 * i], ctx->tev[2 * i + 1]));
    }
    ctx->tcount = 0;
    return n;
}

int vkv_step_run(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, float* key, float* ub,
                 int32_t* sel, double* theta, int32_t* adm, int32_t* adm_count, int64_t cap, float cert_mult,
                 float scale, uint16_t* out, float* lse, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    const bool two_tier = adm_count != nullptr;
    float* ubp = two_tier ? ub : nullptr;
    int rc;
    if ((rc = check_score(ctx, st, ws, ws_bytes, ubp, cert_mult))) return rc;
    if ((rc = check_select(ctx, st, ws, ws_bytes, k, sel, theta))) return rc;
    if (two_tier && (rc = check_admit(ctx, st, ws, ws_bytes, k, sel, theta, ub, cert_mult, adm, adm_count, cap)))
        return rc;
    const int64_t acap = two_tier ? cap : 0;
    if ((rc = check_attend(ctx, st, ws, ws_bytes, k, sel, two_tier ? adm : nullptr, two_tier ? adm_count : nullptr,
                           acap, scale, out, lse)))
        return rc;
    hipStream_t s = (hipStream_t)stream;
    char* w = (char*)ws;
    const Chunk all{0, st->B};
    HIP_TRY(ctx, run_prep(st, w, all, s));
    const bool timed = ctx->timing && ctx->tcount < TIMING_SLOTS;
    if (timed) HIP_TRY(ctx, hipEventRecord(ctx->tev[2 * ctx->tcount], s));
    HIP_TRY(ctx, run_score(st, w, all, key, ubp, cert_mult, s));
    if (timed) HIP_TRY(ctx, hipEventRecord(ctx->tev[2 * ctx->tcount++ + 1], s));
    HIP_TRY(ctx, run_select(st, w, all, k, sel, theta, s));
    if (two_tier) HIP_TRY(ctx, run_admit(st, w, all, k, sel, theta, ub, cert_mult, adm, adm_count, cap, s));
    HIP_TRY(ctx, run_attend(st, w, all, k, sel, two_tier ? adm : nullptr, two_tier ? adm_count : nullptr, acap,
                            scale, out, lse, s));
    if ((rc = debug_check_sel(ctx, st, k, sel, s))) return rc;
    if (two_tier) return debug_check_adm(ctx, st, k, sel, adm, adm_count, cap, s);
    return VKV_OK;
}

static hipError_t run_row_max(const vkv_step* st, const int32_t* rows, int64_t nrows, int all_archive, int add_recent,
                              double* smax, int32_t* argmax, hipStream_t s, char* ws = nullptr) {
    RowMaxArgs a{};
    // with a workspace: row ranges in parallel, about one workgroup per CU in
    // all (a workgroup holds 8 head groups of 16), at least 64 rows each
    a.nsplit = 1;
    if (ws) {
        const int64_t N = (all_archive ? st->T - st->W : nrows) + (add_recent ? st->W : 0);
        const int64_t blocks = ((st->H + 127) / 128) * st->B;
        int64_t ns = std::max<int64_t>(1, (256 + blocks - 1) / std::max<int64_t>(blocks, 1));
        ns = std::min<int64_t>({ns, (int64_t)RM_MAX_SPLIT, std::max<int64_t>(1, N / 64)});
        a.nsplit = (int)ns;
        const WsLayout L = layout(st, 0, 0);
        a.part_v = reinterpret_cast<double*>(ws + L.rmx);
        a.part_u = reinterpret_cast<int32_t*>(ws + L.rmx + (size_t)(st->B * st->H * RM_MAX_SPLIT * 8));
    }
    a.q_lat = st->q_lat;
    a.q_rope = st->q_rope;
    a.cache = st->cache;
    a.cs = st->cache_row_stride;
    a.cbs = st->cache_batch_stride;
    a.rows = rows;
    a.nrows = all_archive ? 0 : nrows;
    a.A = st->T - st->W;
    a.T = st->T;
    a.all_archive = all_archive;
    a.add_recent = add_recent;
    a.B = (int)st->B;
    a.H = (int)st->H;
    a.smax = smax;
    a.argmax = argmax;
    return launch_row_max(a, s);
}

int vkv_row_max(vkv_ctx* ctx, const vkv_step* st, const int32_t* rows, int64_t nrows, int32_t add_recent,
                double* smax, int32_t* argmax, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_step(ctx, st);
    if (rc) return rc;
    if (!smax || !argmax) return fail(ctx, VKV_E_ARG, "smax and argmax are required");
    if (rows && (nrows < 0 || nrows > st->T - st->W))
        return fail(ctx, VKV_E_ARG, "nrows=%lld outside [0, A]", (long long)nrows);
    HIP_TRY(ctx, run_row_max(st, rows, nrows, rows ? 0 : 1, add_recent ? 1 : 0, smax, argmax, (hipStream_t)stream));
    return VKV_OK;
}

static int check_trigger(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, const int32_t* sel,
                         const float* ub, float cert_mult, const double* smax, int64_t topj, int32_t* fired,
                         int32_t* fired_count, int64_t cap) {
    int rc = check_prep(ctx, st, ws, ws_bytes);
    if (rc) return rc;
    if ((rc = check_cert_mult(ctx, cert_mult))) return rc;
    const int64_t A = st->T - st->W;
    if (st->mode == VKV_MODE_DIGEST) return fail(ctx, VKV_E_UNSUPPORTED, "the trigger needs the branch summand in the key");
    if (!st->eta || !st->eps || !st->gam) return fail(ctx, VKV_E_ARG, "the trigger needs eta, eps and gam");
    if (k < 0 || k > A) return fail(ctx, VKV_E_ARG, "k=%lld outside [0, A]", (long long)k);
    if (cap < 0 || cap > A) return fail(ctx, VKV_E_ARG, "cap=%lld outside [0, A]", (long long)cap);
    if (topj < 0) return fail(ctx, VKV_E_ARG, "topj must be >= 0 (0 = uncapped)");
    if (!smax || !fired_count || (A > 0 && !ub) || (cap > 0 && !fired) || (k > 0 && !sel))
        return fail(ctx, VKV_E_ARG, "sel, ub, smax, fired and fired_count are required");
    return VKV_OK;
}

static hipError_t run_trigger(const vkv_step* st, char* w, int64_t k, const int32_t* sel, const float* ub,
                              float cert_mult, const double* smax, int64_t topj, int32_t* fired,
                              int32_t* fired_count, int64_t cap, hipStream_t s) {
    const WsLayout L = layout(st, 0, 0);
    SelectArgs a = select_args(st, L, w, Chunk{0, st->B});
    a.ub = ub;
    a.sel = const_cast<int32_t*>(sel);
    a.adm = fired;
    a.adm_count = fired_count;
    a.k = k;
    a.cap = cap;
    a.cert_mult = cert_mult;
    a.smax = smax;
    a.topj = topj;
    return launch_trigger(a, s);
}

int vkv_trigger(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, const int32_t* sel,
                const float* ub, float cert_mult, const double* smax, int64_t topj, int32_t* fired,
                int32_t* fired_count, int64_t cap, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_trigger(ctx, st, ws, ws_bytes, k, sel, ub, cert_mult, smax, topj, fired, fired_count, cap);
    if (rc) return rc;
    HIP_TRY(ctx, run_trigger(st, (char*)ws, k, sel, ub, cert_mult, smax, topj, fired, fired_count, cap,
                             (hipStream_t)stream));
    return debug_check_adm(ctx, st, k, sel, fired, fired_count, cap, (hipStream_t)stream);
}

int vkv_required_inflation(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, const int32_t* sel,
                           const double* tier1_max, const int32_t* argmax, int32_t* hard, double* zq, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_prep(ctx, st, ws, ws_bytes);
    if (rc) return rc;
    const int64_t A = st->T - st->W;
    if (st->mode == VKV_MODE_DIGEST) return fail(ctx, VKV_E_UNSUPPORTED, "the inflation needs the branch summand in the key");
    if (!st->eta || !st->eps || !st->gam) return fail(ctx, VKV_E_ARG, "the inflation needs eta, eps and gam");
    if (k < 0 || k > A) return fail(ctx, VKV_E_ARG, "k=%lld outside [0, A]", (long long)k);
    if (!tier1_max || !argmax || !hard || !zq || (k > 0 && !sel))
        return fail(ctx, VKV_E_ARG, "sel, tier1_max, argmax, hard and zq are required");
    const WsLayout L = layout(st, 0, 0);
    InflArgs a{};
    index_operand(st, &a.x, &a.xs, &a.xbs);
    a.qt = reinterpret_cast<const uint16_t*>((char*)ws + L.qt);
    a.hsc = reinterpret_cast<const float*>((char*)ws + L.hsc);
    a.eta = st->eta;
    a.eps = st->eps;
    a.gam = st->gam;
    a.T = st->T;
    a.A = A;
    a.k = k;
    a.sel = sel;
    a.tier1 = tier1_max;
    a.argmax = argmax;
    a.B = (int)st->B;
    a.H = (int)st->H;
    a.n = (int)L.n;
    a.r = (st->mode & 2) ? st->r : 0;
    a.hard = hard;
    a.zq = zq;
    HIP_TRY(ctx, launch_inflation(a, (hipStream_t)stream));
    return VKV_OK;
}

int vkv_conformal_z(const double* zq, int64_t n, int64_t tau_num, int64_t tau_den, double zmax, double* z,
                    int64_t* min_hard, int64_t* rank) {
    if (!z || !min_hard || !rank || (n > 0 && !zq) || n < 0) return fail(nullptr, VKV_E_ARG, "bad arguments");
    if (tau_num <= 0 || tau_den <= tau_num) return fail(nullptr, VKV_E_ARG, "tau = tau_num / tau_den must lie in (0, 1)");
    if (!(zmax >= 0.0)) return fail(nullptr, VKV_E_ARG, "zmax must be >= 0");
    // tau_s = 2 tau_num / (tau_den + tau_num); min_hard = ceil(tau_s / (1 - tau_s)); k = ceil((n + 1) tau_s)
    const int64_t mh = (2 * tau_num + (tau_den - tau_num) - 1) / (tau_den - tau_num);
    const int64_t k = ((n + 1) * 2 * tau_num + (tau_den + tau_num) - 1) / (tau_den + tau_num);
    *min_hard = mh;
    if (n < mh || k > n) {
        *z = zmax;
        *rank = 0;
        return VKV_OK;
    }
    std::vector<double> v(zq, zq + n);
    std::nth_element(v.begin(), v.begin() + (k - 1), v.end());
    double q = v[(size_t)(k - 1)];
    if (q > zmax) q = zmax;
    if (!(q > 0.0)) q = 0.0;
    *z = q;
    *rank = k;
    return VKV_OK;
}

int vkv_step_run_trigger(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, float* key, float* ub,
                         int32_t* sel, double* theta, float cert_mult, double* smax, int32_t* argmax, int64_t topj,
                         int32_t* fired, int32_t* fired_count, int64_t cap, float scale, uint16_t* out, float* lse,
                         void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc;
    if ((rc = check_score(ctx, st, ws, ws_bytes, ub, cert_mult))) return rc;
    if (!ub) return fail(ctx, VKV_E_ARG, "the trigger needs ub");
    if ((rc = check_select(ctx, st, ws, ws_bytes, k, sel, theta))) return rc;
    if ((rc = check_trigger(ctx, st, ws, ws_bytes, k, sel, ub, cert_mult, smax, topj, fired, fired_count, cap)))
        return rc;
    if (!argmax) return fail(ctx, VKV_E_ARG, "argmax is required");
    if ((rc = check_attend(ctx, st, ws, ws_bytes, k, sel, fired, fired_count, cap, scale, out, lse))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char* w = (char*)ws;
    const Chunk all{0, st->B};
    HIP_TRY(ctx, run_prep(st, w, all, s));
    HIP_TRY(ctx, run_score(st, w, all, key, ub, cert_mult, s));
    HIP_TRY(ctx, run_select(st, w, all, k, sel, theta, s));
    // the tier-1 maximum logit per head over S and the recent window
    HIP_TRY(ctx, run_row_max(st, sel, k, 0, 1, smax, argmax, s, w));
    HIP_TRY(ctx, run_trigger(st, w, k, sel, ub, cert_mult, smax, topj, fired, fired_count, cap, s));
    HIP_TRY(ctx, run_attend(st, w, all, k, sel, fired, fired_count, cap, scale, out, lse, s));
    if ((rc = debug_check_sel(ctx, st, k, sel, s))) return rc;
    return debug_check_adm(ctx, st, k, sel, fired, fired_count, cap, s);
}

int vkv_sigma_workspace_size(int64_t B, int64_t nblk, size_t* bytes) {
    if (!bytes) return fail(nullptr, VKV_E_ARG, "bytes is NULL");
    if (B < 0 || nblk < 0 || B > 65535 || nblk > 65535) return fail(nullptr, VKV_E_SHAPE, "B or nblk out of range");
    *bytes = up256(sigma_workspace_bytes(B, nblk));
    return VKV_OK;
}

int vkv_sigma_close(vkv_ctx* ctx, const uint16_t* cache, int64_t B, int64_t T, int64_t cache_row_stride,
                    int64_t cache_batch_stride, int64_t t0, int64_t nblk, int32_t kappa, void* ws, size_t ws_bytes,
                    double* sigma, int64_t sigma_stride, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    if (!cache) return fail(ctx, VKV_E_ARG, "cache is NULL");
    if (B < 1 || B > 65535 || T < 1 || T >= (1ll << 31)) return fail(ctx, VKV_E_SHAPE, "B=%lld T=%lld", (long long)B, (long long)T);
    if (!al16(cache) || cache_row_stride < D_ROW || cache_row_stride % 8 || cache_batch_stride % 8 ||
        (B > 1 && cache_batch_stride < T * cache_row_stride))
        return fail(ctx, VKV_E_ALIGN, "cache strides");
    if (t0 < 0 || t0 % VKV_SIGMA_BLOCK || nblk < 0 || nblk > 65535 || t0 + nblk * VKV_SIGMA_BLOCK > T)
        return fail(ctx, VKV_E_SHAPE, "t0=%lld nblk=%lld: blocks of %d rows from a multiple of %d, within T=%lld",
                    (long long)t0, (long long)nblk, VKV_SIGMA_BLOCK, VKV_SIGMA_BLOCK, (long long)T);
    if (kappa < 1 || kappa > VKV_SIGMA_BLOCK / 2) return fail(ctx, VKV_E_ARG, "kappa=%d outside [1, %d]", kappa, VKV_SIGMA_BLOCK / 2);
    if (nblk == 0) return VKV_OK;
    if (!sigma || ((uintptr_t)sigma & 7u)) return fail(ctx, VKV_E_ARG, "sigma must be an 8-byte aligned device pointer");
    if (sigma_stride < t0 + nblk * VKV_SIGMA_BLOCK) return fail(ctx, VKV_E_ARG, "sigma_stride smaller than the closed rows");
    int rc = check_ws(ctx, ws, ws_bytes, up256(sigma_workspace_bytes(B, nblk)));
    if (rc) return rc;
    SigmaArgs a{};
    a.cache = cache;
    a.crs = cache_row_stride;
    a.cbs = cache_batch_stride;
    a.t0 = t0;
    a.nblk = nblk;
    a.kappa = kappa;
    a.B = (int)B;
    a.part = reinterpret_cast<double*>(ws);
    a.sigma = sigma;
    a.sstride = sigma_stride;
    HIP_TRY(ctx, launch_sigma(a, (hipStream_t)stream));
    return VKV_OK;
}

int vkv_sigma_select(vkv_ctx* ctx, const double* sigma, int64_t B, int64_t n_closed, int64_t sigma_stride, int64_t m,
                     int32_t nsink, int32_t* kept, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    if (B < 1 || B > 65535 || n_closed < 0 || n_closed >= (1ll << 31)) return fail(ctx, VKV_E_SHAPE, "B or n_closed out of range");
    if (m < 0 || nsink < 0) return fail(ctx, VKV_E_ARG, "m and nsink must be >= 0");
    const int64_t lo = std::min<int64_t>(nsink, n_closed);
    const int64_t K = lo + std::min<int64_t>(m, n_closed - lo);
    if (K == 0) return VKV_OK;
    if (!sigma || !kept || ((uintptr_t)sigma & 7u)) return fail(ctx, VKV_E_ARG, "sigma and kept are required");
    if (sigma_stride < n_closed) return fail(ctx, VKV_E_ARG, "sigma_stride smaller than n_closed");
    SigmaSelArgs a{};
    a.sigma = sigma;
    a.sstride = sigma_stride;
    a.n = n_closed;
    a.m = m;
    a.nsink = nsink;
    a.kept = kept;
    a.kstride = K;
    a.B = (int)B;
    HIP_TRY(ctx, launch_sigma_select(a, (hipStream_t)stream));
    return VKV_OK;
}

int vkv_step_run_kept(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k, const int32_t* kept,
                      float* key, float* ub, float cert_mult, double* smax, int32_t* argmax, int64_t topj,
                      int32_t* fired, int32_t* fired_count, int64_t cap, float scale, uint16_t* out, float* lse,
                      void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc;
    if ((rc = check_score(ctx, st, ws, ws_bytes, ub, cert_mult))) return rc;
    if (!ub) return fail(ctx, VKV_E_ARG, "the trigger needs ub");
    if ((rc = check_trigger(ctx, st, ws, ws_bytes, k, kept, ub, cert_mult, smax, topj, fired, fired_count, cap)))
        return rc;
    if (!argmax) return fail(ctx, VKV_E_ARG, "argmax is required");
    if ((rc = check_attend(ctx, st, ws, ws_bytes, k, kept, fired, fired_count, cap, scale, out, lse))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char* w = (char*)ws;
    const Chunk all{0, st->B};
    const WsLayout L = layout(st, k, cap);
    // the tier's maximum logit does not depend on the scan, so it comes first
    // and the scan writes the trigger margins max_h (UB~_h - s*_h) directly
    HIP_TRY(ctx, run_prep(st, w, all, s));
    HIP_TRY(ctx, launch_mark_tier(reinterpret_cast<uint8_t*>(w + L.flags), flag_stride(L.A), L.A, (int)st->B, kept, k, s));
    HIP_TRY(ctx, run_row_max(st, kept, k, 0, 1, smax, argmax, s, w));
    // the step reads only the margins: without a key buffer the scan writes no keys
    HIP_TRY(ctx, run_score(st, w, all, key, ub, cert_mult, s, smax, key == nullptr));
    HIP_TRY(ctx, run_trigger(st, w, k, kept, ub, cert_mult, smax, topj, fired, fired_count, cap, s));
    HIP_TRY(ctx, run_attend(st, w, all, k, kept, fired, fired_count, cap, scale, out, lse, s));
    if ((rc = debug_check_sel(ctx, st, k, kept, s))) return rc;
    return debug_check_adm(ctx, st, k, kept, fired, fired_count, cap, s);
}

int vkv_pack_rows(vkv_ctx* ctx, const int32_t* lists, const int32_t* counts, int64_t n, int64_t cap,
                  int32_t* offsets, int32_t* packed, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    if (n < 0 || n > 65535 || cap < 0 || n * cap >= (1ll << 31)) return fail(ctx, VKV_E_SHAPE, "n or cap out of range");
    if (!offsets || (n > 0 && !counts) || (n > 0 && cap > 0 && (!lists || !packed)))
        return fail(ctx, VKV_E_ARG, "lists, counts, offsets and packed are required");
    HIP_TRY(ctx, launch_pack_rows(lists, counts, n, cap, offsets, packed, (hipStream_t)stream));
    return VKV_OK;
}

static int check_page(vkv_ctx* ctx, const vkv_step* st, int64_t page) {
    int rc = check_step(ctx, st);
    if (rc) return rc;
    if (page < 1 || page > (1ll << 30)) return fail(ctx, VKV_E_ARG, "page=%lld outside [1, 2^30]", (long long)page);
    return VKV_OK;
}

static PageArgs page_args(const vkv_step* st, int64_t page) {
    PageArgs a{};
    index_operand(st, &a.x, &a.xs, &a.xbs);
    a.A = st->T - st->W;
    a.page = page;
    a.npages = (a.A + page - 1) / page;
    a.n = index_width(st);
    a.H = (int)st->H;
    a.B = (int)st->B;
    return a;
}

int vkv_page_box(vkv_ctx* ctx, const vkv_step* st, int64_t page, uint16_t* box, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_page(ctx, st, page);
    if (rc) return rc;
    PageArgs a = page_args(st, page);
    if (a.npages == 0) return VKV_OK;   // no archived rows
    if (!box) return fail(ctx, VKV_E_ARG, "box is required");
    if (!al16(box)) return fail(ctx, VKV_E_ALIGN, "box must be 16-byte aligned");
    a.box = box;
    HIP_TRY(ctx, launch_page_box(a, (hipStream_t)stream));
    return VKV_OK;
}

int vkv_page_bound(vkv_ctx* ctx, const vkv_step* st, const void* ws, size_t ws_bytes, int64_t page,
                   const uint16_t* box, double* bound, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_prep(ctx, st, const_cast<void*>(ws), ws_bytes);
    if (rc) return rc;
    if ((rc = check_page(ctx, st, page))) return rc;
    PageArgs a = page_args(st, page);
    if (a.npages == 0) return VKV_OK;   // no archived rows
    if (!box || !bound) return fail(ctx, VKV_E_ARG, "box and bound are required");
    if (!al16(box)) return fail(ctx, VKV_E_ALIGN, "box must be 16-byte aligned");
    a.box = const_cast<uint16_t*>(box);
    a.qt = reinterpret_cast<const uint16_t*>((const char*)ws + layout(st, 0, 0).qt);
    a.bound = bound;
    HIP_TRY(ctx, launch_page_bound(a, (hipStream_t)stream));
    return VKV_OK;
}

int vkv_sketch_workspace_size(int32_t r, size_t* bytes) {
    if (!bytes) return fail(nullptr, VKV_E_ARG, "bytes is NULL");
    if (r < 32 || r > 512 || r % 32) return fail(nullptr, VKV_E_UNSUPPORTED, "r=%d: need a multiple of 32 in [32, 512]", r);
    *bytes = up256(sketch_workspace_bytes(r));
    return VKV_OK;
}

int vkv_sketch_basis(vkv_ctx* ctx, const uint16_t* q, int64_t m, int32_t r, int32_t iters, void* ws, size_t ws_bytes,
                     uint16_t* P, double* energy, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    if (!q || !P) return fail(ctx, VKV_E_ARG, "q and P are required");
    if (m < 1) return fail(ctx, VKV_E_SHAPE, "m=%lld: need at least one query", (long long)m);
    if (r < 32 || r > 512 || r % 32) return fail(ctx, VKV_E_UNSUPPORTED, "r=%d: need a multiple of 32 in [32, 512]", r);
    if (iters < 0 || iters > 64) return fail(ctx, VKV_E_ARG, "iters=%d outside [0, 64]", iters);
    if (!al16(q) || !al16(P)) return fail(ctx, VKV_E_ALIGN, "q and P must be 16-byte aligned");
    int rc = check_ws(ctx, ws, ws_bytes, up256(sketch_workspace_bytes(r)));
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(ctx, launch_sketch(q, m, r, iters, ws, P, energy, s));
    // the orthonormalisation's verdict (one int at the end of the workspace)
    int bad = 0;
    const size_t off = sketch_workspace_bytes(r) - 256;
    HIP_TRY(ctx, hipMemcpyAsync(&bad, (char*)ws + off, sizeof(int), hipMemcpyDeviceToHost, s));
    HIP_TRY(ctx, hipStreamSynchronize(s));
    if (bad) return fail(ctx, VKV_E_UNSUPPORTED, "the queries span fewer than r=%d dimensions", r);
    return VKV_OK;
}

int vkv_step_run_static(vkv_ctx* ctx, const vkv_step* st, int64_t k, float* key, float* ub, int32_t* sel,
                        double* theta, int32_t* adm, int32_t* adm_count, int64_t cap, float cert_mult, float scale,
                        uint16_t* out, float* lse, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_step(ctx, st);
    if (rc) return rc;
    const int64_t A = st->T - st->W;
    if (k < 0 || k > A) return fail(ctx, VKV_E_ARG, "k=%lld outside [0, A=%lld]", (long long)k, (long long)A);
    const int64_t acap = adm_count ? cap : 0;
    if (acap < 0 || acap > A) return fail(ctx, VKV_E_ARG, "cap=%lld outside [0, A]", (long long)cap);
    const size_t need = layout(st, k, acap).total;
    if (need > (size_t)VKV_STATIC_WS_BYTES)
        return fail(ctx, VKV_E_WORKSPACE,
                    "this step needs a workspace of %zu bytes; vkv_step_run_static has %zu (use vkv_step_run with a "
                    "caller workspace)",
                    need, (size_t)VKV_STATIC_WS_BYTES);
    (void)hipSetDevice(ctx->device);
    return vkv_step_run(ctx, st, ctx->scratch_ptr, (size_t)VKV_STATIC_WS_BYTES, k, key, ub, sel, theta, adm, adm_count,
                        cap, cert_mult, scale, out, lse, stream);
}

int vkv_check_rows(vkv_ctx* ctx, const vkv_step* st, int64_t k, const int32_t* sel, const int32_t* adm,
                   const int32_t* adm_count, int64_t cap, void* stream) {
    if (!ctx) return fail(nullptr, VKV_E_ARG, "ctx is NULL");
    int rc = check_step(ctx, st);
    if (rc) return rc;
    const int64_t A = st->T - st->W;
    if (k < 0 || k > A) return fail(ctx, VKV_E_ARG, "k=%lld outside [0, A]", (long long)k);
    if (cap < 0 || cap > A) return fail(ctx, VKV_E_ARG, "cap=%lld outside [0, A]", (long long)cap);
    if ((k > 0 && !sel) || (cap > 0 && !adm)) return fail(ctx, VKV_E_ARG, "sel and adm are required");
    hipStream_t s = (hipStream_t)stream;
    const int saved = ctx->debug_rows;
    ctx->debug_rows = 1;
    rc = debug_check_sel(ctx, st, k, sel, s);
    if (!rc && adm_count) rc = debug_check_adm(ctx, st, k, sel, adm, adm_count, cap, s);
    ctx->debug_rows = saved;
    return rc;
}

}  // extern "C"
