// vkv_internal.h -- shared declarations of the libvkv HIP sources (gfx950).
//
// Device helpers for bit-exact fp64 -> bf16 rounding, upward roundings used by
// the certificate scalars, the order-preserving key encoding of the radix
// select, and the launch interfaces of the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/vkv.h"

namespace vkv {

constexpr int D_LAT = 512;
constexpr int D_ROPE = 64;
constexpr int D_ROW = 576;

// Margin that turns fp64 norm computations into rigorous upper bounds:
// 2^-40 exceeds 16x the worst relative error of a 512-term fp64 dot product.
constexpr double CERT_G = 0x1p-40;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint16_t u16x8_t __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------ bit casts

__host__ __device__ __forceinline__ uint32_t f2u(float f) { return __builtin_bit_cast(uint32_t, f); }
__host__ __device__ __forceinline__ float u2f(uint32_t u) { return __builtin_bit_cast(float, u); }
__host__ __device__ __forceinline__ uint64_t d2u(double d) { return __builtin_bit_cast(uint64_t, d); }
__host__ __device__ __forceinline__ double u2d(uint64_t u) { return __builtin_bit_cast(double, u); }

// ------------------------------------------------------------ bf16 helpers

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// fp32 -> bf16, round to nearest even (finite inputs; NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x0040u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// fp64 -> bf16 in a single round-to-nearest-even step, by integer arithmetic
// on the fp64 significand (no intermediate fp32 rounding).
__host__ __device__ __forceinline__ uint16_t f64_to_bf16_rne(double x) {
    uint64_t u = d2u(x);
    uint16_t sign = (uint16_t)((u >> 48) & 0x8000u);
    uint64_t ax = u & 0x7FFFFFFFFFFFFFFFull;
    if (ax > 0x7FF0000000000000ull) return 0x7FC0;          // NaN
    if (ax == 0x7FF0000000000000ull) return sign | 0x7F80;   // inf
    int be = (int)(ax >> 52);
    if (be == 0) return sign;                                // fp64 subnormal: far below bf16
    int E = be - 1023;
    if (E > 127) return sign | 0x7F80;
    if (E < -134) return sign;
    uint64_t m = (ax & 0x000FFFFFFFFFFFFFull) | 0x0010000000000000ull;
    int shift = (E >= -126) ? 45 : (-81 - E);                // bits below the bf16 quantum
    uint64_t q = m >> shift;
    uint64_t rem = m & ((1ull << shift) - 1ull);
    uint64_t half = 1ull << (shift - 1);
    if (rem > half || (rem == half && (q & 1ull))) q += 1ull;
    uint32_t bits = (E >= -126) ? (uint32_t)(((E + 127) << 7) + (int)(q - 128ull)) : (uint32_t)q;
    if (bits > 0x7F80u) bits = 0x7F80u;
    return (uint16_t)(sign | bits);
}

// ------------------------------------------------------- upward roundings

__host__ __device__ __forceinline__ float next_up_f32(float f) {
    uint32_t b = f2u(f);
    if ((b & 0x7FFFFFFFu) >= 0x7F800000u) return f;          // inf / nan
    if ((b & 0x7FFFFFFFu) == 0u) return u2f(1u);  // +-0 -> min subnormal
    return u2f((b & 0x80000000u) ? b - 1u : b + 1u);
}

__host__ __device__ __forceinline__ float next_down_f32(float f) { return -next_up_f32(-f); }

// Smallest float f with (double)f >= x.
__host__ __device__ __forceinline__ float ru_f32(double x) {
    float f = (float)x;
    if ((double)f < x) f = next_up_f32(f);
    return f;
}

// Smallest float f >= 0 with f*f >= x, decided with exact fp64 products.
__host__ __device__ __forceinline__ float ru_sqrt_f32(double x) {
    if (!(x > 0.0)) return 0.0f;
    if (!(x < 0x1.fffffep+127 * 0x1.fffffep+127)) return u2f(0x7F800000u);   // beyond FLT_MAX^2
    float f = (float)sqrt(x);                                // within an ulp of the answer
    while ((double)f * (double)f < x) f = next_up_f32(f);
    while (f > 0.0f) {
        float p = u2f(f2u(f) - 1u);
        if ((double)p * (double)p >= x) f = p;
        else break;
    }
    return f;
}

// Order-preserving map float -> uint32 (larger float -> larger uint).
__host__ __device__ __forceinline__ uint32_t key_to_ord(float f) {
    uint32_t u = f2u(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__host__ __device__ __forceinline__ float ord_to_key(uint32_t o) {
    uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
    return u2f(u);
}

// ----------------------------------------------------------- workspace

// Per-sequence state words (uint32 each), kept in the workspace.  Words 0-7
// are the scorer's (cleared by the query prep of the step); the others are
// written, never accumulated, by the selection and admission calls, so those
// calls may be repeated on the same workspace.
enum SeqWord : int {
    SQ_QMAX = 0,    // float bits: max_h ||qt_h|| (upper bound)
    SQ_NU2MAX = 1,  // float bits: max_u ||x_u||^2 (fp32 sum)
    SQ_BMAX = 2,    // float bits: max_u (amax eta + nmax eps + emax gam)
    SQ_AMAX = 3,    // float bits: max_h a'_h, n_h, e_h (written by the scorer launch)
    SQ_NMAX = 4,
    SQ_EMAX = 5,
    SQ_KMIN = 6,    // ordered encoding of min_u key~_u   (scorer, atomicMin)
    SQ_KMAX = 7,    // ordered encoding of max_u key~_u   (scorer, atomicMax)
    SQ_BLO = 8,     // float bits: lower end of the sampled bracket of the k-th key~
    SQ_BHI = 9,     // float bits: upper end of the sampled bracket
    SQ_CLO = 10,    // float bits: rows with key~ + E below this are certainly not selected
    SQ_CHI = 11,    // float bits: rows with key~ - E above this are certainly selected
    SQ_CMULT = 12,  // float bits: the certificate multiplier the scorer's bound used
    SQ_TLO = 13,    // float bits: LO <= k-th largest of (key~ - E)   (diagnostic)
    SQ_THI = 14,    // float bits: HI >= k-th largest of (key~ + E)   (diagnostic)
    SQ_NAMB = 15,   // ambiguous rows of the selection                (diagnostic)
    SQ_NAMB2 = 16,  // ambiguous rows of the admission                (diagnostic)
    SQ_NCAND = 17,  // selection candidates listed by the counting pass (zeroed by the bracket launch)
    SQ_NCAND2 = 18, // undecided admission rows listed by the classification (zeroed by its consumer)
    SQ_NCAND3 = 19, // trigger candidates listed by the trigger classification (zeroed by its consumer)
    SQ_NFIRED = 20, // rows the trigger fired before the top-j cap (diagnostic)
    SQ_TRGM = 21,   // 1: the scorer's ub holds trigger margins max_h (UB~_h - s*_h)
    SQ_WORDS = 32
};

constexpr int CB_KEYS = 4096;      // archive rows per counting / classification block
constexpr int BLK_WORDS = 4;       // per counting block: the counts below
// per counting block: rows it decided in (selected / admitted), rows above the
// sampled bracket, and rows of its range the resolve block decided in
enum BlockWord : int { BW_IN = 0, BW_XIN = 1, BW_ABOVE = 2 };
constexpr int HIST_BINS = 4096;
constexpr int ATT_CHUNK = 32;      // rows per attention tile
constexpr int ATT_HEADS = 128;     // heads per attention workgroup (8 waves x 16)
constexpr int ATT_MAX_SPLIT_ROWS = 1024;   // rows of one split (row list held in LDS)

struct WsLayout {
    size_t qt, hsc, seq, kt, flags, flags2, blk, cand, candkey, amb, ambkey, rmx, part_o, part_ml, total;
    int64_t A, n, nblk, splits, rows_per_split, base_splits, rows_per_adm, adm_blocks, cap;
};

// ------------------------------------------------------ kernel interfaces

struct QprepArgs {
    const uint16_t* q_lat;
    const uint16_t* q_rope;
    const uint16_t* P;
    int B, H, r, mode, n;
    uint16_t* qt;      // [B,H,n]
    float* hsc;        // [B,H,4]: a, nq, e, ||qt||
    uint32_t* seq;     // [B,SQ_WORDS] (cleared here for the step)
};

struct ScoreArgs {
    const uint16_t* x;     // index rows (already offset to the first scored column)
    int64_t xs, xbs;       // row / batch stride, elements
    const uint16_t* qt;    // [B,H,n]
    const float* hsc;      // [B,H,4]
    const float* eta;      // [B,T] (UB only)
    const float* eps;
    const float* gam;
    int64_t T;
    float* key;            // [B,A] or null (diagnostic)
    float* ub;             // [B,A] or null
    float* kt;             // [B,A]: key~ (fp32 matrix-core index keys)
    uint32_t* seq;
    int64_t A;
    int B, H, n;
    float cert_mult;       // (UB) multiplier of the sketch-residual term a_h eta_u
    const double* thr;     // (UB) [B,H] trigger thresholds s*_h, or null: ub holds max_h (UB~_h - s*_h)
    int no_keys;           // (UB) 1: only ub is written (no key, no kt); the LDS key buffer then holds
                           // bounds only, so a wave owns twice the tiles
};

struct DigestArgs {
    const uint16_t* cache;
    int64_t cs, cbs;
    const uint16_t* P;
    int r, with_rope;
    uint16_t* index;
    int64_t is, ibs;
    float* eta;
    float* eps;
    float* gam;
    int64_t B, T;
};

struct SelectArgs {
    const float* kt;       // [B,A] key~ from the scorer
    const float* ub;       // [B,A] (admit)
    const uint16_t* x;     // index rows for fp64 re-scoring
    int64_t xs, xbs;
    const uint16_t* qt;
    const float* hsc;
    const float* eta;
    const float* eps;
    const float* gam;
    int64_t T;
    uint32_t* seq;
    uint8_t* flags;        // [B,A] selection: 1 selected, 0 not, 2 undecided
    uint8_t* flags2;       // [B,A] admission: 3 admitted, 0 not, 4 undecided
    uint32_t* blk;         // [B,nblk,BLK_WORDS] per counting block
    int32_t* cand;         // [B,A] candidate rows (selection) / undecided rows (admission), listed
    float* candkey;        // [B,A] the candidates' keys~ (selection)
    int32_t* amb;          // [B,A] the undecided rows, compacted
    uint64_t* ambkey;      // [B,A] their exact keys (order-preserving encoding of fp64)
    int32_t* sel;          // [B,k]
    double* theta;         // [B]
    int32_t* adm;          // [B,cap]
    int32_t* adm_count;    // [B]
    int64_t A, k, cap, nblk;
    int64_t fstride;       // bytes per sequence of flags / flags2 (A rounded up to 64)
    int B, H, n;
    float cert_mult;       // admission: multiplier of the sketch-residual term
    const double* smax;    // trigger: [B,H] per-head thresholds s*_h (the tier-1 max logit)
    int64_t topj;          // trigger: cap on the fired rows (0 = uncapped)
};

struct RowMaxArgs {
    const uint16_t* q_lat;  // [B,H,512]
    const uint16_t* q_rope; // [B,H,64]
    const uint16_t* cache;
    int64_t cs, cbs;
    const int32_t* rows;    // [B,nrows] listed rows (unless all_archive)
    int64_t nrows, A, T;
    int all_archive;        // the list is the archived rows [0, A)
    int add_recent;         // the rows [A, T) follow the listed ones
    int B, H;
    double* smax;           // [B,H]
    int32_t* argmax;        // [B,H]
    int nsplit;             // row ranges scanned in parallel (1: no scratch needed)
    double* part_v;         // [B,H,nsplit] per-range maxima (nsplit > 1)
    int32_t* part_u;        // [B,H,nsplit] their rows
};
constexpr int RM_MAX_SPLIT = 16;

struct InflArgs {
    const uint16_t* x;      // index rows
    int64_t xs, xbs;
    const uint16_t* qt;     // [B,H,n]
    const float* hsc;       // [B,H,4]
    const float* eta;
    const float* eps;
    const float* gam;
    int64_t T, A, k;
    const int32_t* sel;     // [B,k]
    const double* tier1;    // [B,H] s*_h
    const int32_t* argmax;  // [B,H] the causal argmax rows
    int B, H, n, r;
    int32_t* hard;          // [B,H]
    double* zq;             // [B,H]
};

struct AttendArgs {
    const uint16_t* q_lat;
    const uint16_t* q_rope;
    const uint16_t* cache;
    int64_t cs, cbs;
    const int32_t* sel;
    const int32_t* adm;
    const int32_t* adm_count;
    int64_t k, W, A, cap;
    int64_t rows_per_split;   // rows of each of the first base_splits splits (kept rows and window)
    int64_t rows_per_adm;     // rows of each later split (the admitted rows' capacity)
    int splits, base_splits;
    int adm_blocks;           // workgroups that take the admitted splits in turn
    int B, H;
    float scale_log2;      // scale * log2(e)
    uint16_t* part_o;      // bf16 [B, splits, head groups, 8 waves, 32, 64 lanes, 4] (register order)
    float* part_ml;        // [B, splits, H, 2]
    uint16_t* out;         // [B,H,512]
    float* lse;            // [B,H]
};

hipError_t launch_qprep(const QprepArgs& a, hipStream_t s);
hipError_t launch_score(const ScoreArgs& a, hipStream_t s);
hipError_t launch_digest(const DigestArgs& a, hipStream_t s);
hipError_t launch_gram_rows(const uint16_t* P, int r, double* rowsum, hipStream_t s);
hipError_t launch_select(const SelectArgs& a, hipStream_t s);
hipError_t launch_admit(const SelectArgs& a, hipStream_t s);
hipError_t launch_attend(const AttendArgs& a, hipStream_t s);
hipError_t launch_row_max(const RowMaxArgs& a, hipStream_t s);
hipError_t launch_trigger(const SelectArgs& a, hipStream_t s);
hipError_t launch_inflation(const InflArgs& a, hipStream_t s);
struct SigmaArgs {
    const uint16_t* cache;
    int64_t crs, cbs;      // cache row / batch strides (elements)
    int64_t t0, nblk;      // first row (a multiple of 4096) and number of blocks to close
    int kappa, B;
    double* part;          // [B, nblk, 8, 4096] squared residuals per channel group
    double* sigma;         // [B, sstride]
    int64_t sstride;
};

struct SigmaSelArgs {
    const double* sigma;
    int64_t sstride, n, m, nsink;
    int32_t* kept;
    int64_t kstride;
    int B;
};

size_t sigma_workspace_bytes(int64_t B, int64_t nblk);
hipError_t launch_sigma(const SigmaArgs& a, hipStream_t s);
hipError_t launch_sigma_select(const SigmaSelArgs& a, hipStream_t s);
// page boxes and interval bounds (page-bound pruning)
struct PageArgs {
    const uint16_t* x;     // index rows as the scorer reads them (first scored column)
    int64_t xs, xbs;       // row / batch stride, elements
    int64_t A, page, npages;
    int n, H, B;
    uint16_t* box;         // [B][npages][2][n]: lo row, hi row (bf16 bits)
    const uint16_t* qt;    // [B][H][n]
    double* bound;         // [B][npages]
};
hipError_t launch_page_box(const PageArgs& a, hipStream_t s);
hipError_t launch_page_bound(const PageArgs& a, hipStream_t s);

hipError_t launch_mark_tier(uint8_t* flags, int64_t fstride, int64_t A, int B, const int32_t* sel, int64_t k,
                            hipStream_t s);

hipError_t launch_pack_rows(const int32_t* lists, const int32_t* counts, int64_t n, int64_t cap, int32_t* offsets,
                            int32_t* packed, hipStream_t s);

size_t sketch_workspace_bytes(int r);
hipError_t launch_sketch(const uint16_t* q, int64_t m, int r, int iters, void* ws, uint16_t* P, double* energy,
                         hipStream_t s);

// ------------------------------------------- fp64 matrix-core row products

typedef double f64x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double bf16_bits_f64(uint16_t v) { return (double)__uint_as_float((uint32_t)v << 16); }

// One 16x16 tile of fp64 row products over 512 dims, i ascending:
//   D[m][n] = sum_{i<512} A[m][i] B[n][i]
// with A, B rows of bf16 staged in LDS.  v_mfma_f64_16x16x4f64 adds its four
// products (k = 0..3) to the accumulator one after another, each with one
// rounding, so 128 of them in i order give the sequential fp64 sum (bf16
// products are exact in fp64).  pa / pb point at element lane / 16 of this
// lane's A row (lane mod 16) and B row; step s reads element 4 s of each.
// Result: lane l, element e = D[4 e + l / 16][l mod 16].  With WN the vector
// unit also accumulates n2 += x^2 over pn[0..512) in order (one fp64 FMA per
// element, between the matrix steps).  The operand reads of each group of 4
// steps are issued one group ahead (scheduling barriers keep them there; at
// most 10 reads are then younger than the awaited ones, within the range of
// an lgkmcnt wait).
template <bool WN>
__device__ __forceinline__ f64x4_t mfma_f64_rowdot512(const uint16_t* pa, const uint16_t* pb, const uint16_t* pn,
                                                      double& n2) {
    constexpr int G = 4, NG = 512 / 4 / G;
    f64x4_t acc = f64x4_t{0.0, 0.0, 0.0, 0.0};
    uint16_t ra[2][G], rb[2][G];
    u16x8_t rn[2][G / 2];
    auto load = [&](int g, int buf) {
#pragma unroll
        for (int e = 0; e < G; ++e) {
            ra[buf][e] = pa[4 * (G * g + e)];
            rb[buf][e] = pb[4 * (G * g + e)];
        }
        if constexpr (WN) {
#pragma unroll
            for (int e = 0; e < G / 2; ++e) rn[buf][e] = *reinterpret_cast<const u16x8_t*>(pn + 4 * G * g + 8 * e);
        }
    };
    load(0, 0);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        if (g + 1 < NG) load(g + 1, (g + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
        const int buf = g & 1;
#pragma unroll
        for (int e = 0; e < G; ++e) {
            acc = __builtin_amdgcn_mfma_f64_16x16x4f64(bf16_bits_f64(ra[buf][e]), bf16_bits_f64(rb[buf][e]), acc, 0, 0,
                                                      0);
            if constexpr (WN) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const double x = bf16_bits_f64(rn[buf][e / 2][4 * (e & 1) + k]);
                    n2 = fma(x, x, n2);
                }
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    return acc;
}

}  // namespace vkv
