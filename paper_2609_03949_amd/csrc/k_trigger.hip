// k_trigger.hip -- the tier-1 maximum logit and the calibration statistic of
// the calibrated trigger (Sec. 4.2: Eq. (trigger), the z paragraph; Sec. 5.2).
//
// row_max_kernel: per sequence b and head h, the maximum over a row list of
// the exact full score s_h(u) = q_lat_h . c_u + q_rope_h . r_u (Sec. 3,
// Eq. (setup); the fp64 sum over the 576 dims, latent then branch, from +0)
// and the row attaining it (ties: the lower row index).  Over the tier-1
// rows it is the trigger threshold s*_h; over the whole context it is the
// causal argmax row of a calibration query.  A workgroup of 8 waves (16
// heads each) streams one range of the list through an LDS tile ring that all
// its waves read: bf16 MFMA scores in fp32 with a per-(row, head) certified
// band e = 2 (n + n/32) 2^-23 ||q_h|| ||x_u|| (n = 576, the scan's error
// model), a running certified lower bound M_h of the maximum, and in LDS the
// rows whose upper bound reaches M_h.  Only those get the fp64 chain; the
// true maximum row always does.  The ranges' maxima are merged by
// row_merge_kernel.
//
// inflation_kernel: for each (calibration query, head), whether the causal
// argmax row is archived and outside the tier-1 set (a hard query), and then
// z_q = (s*_h - idx_h(u*)) / cert_h(u*), the inflation at which the trigger
// score reaches the tier-1 maximum.
#include "vkv_internal.h"

namespace vkv {

constexpr int RM_CAND = 64;           // candidate rows kept per head
constexpr int RM_KS = D_ROW / 32;     // 18 k-steps of the 576-dim score

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float sumsq8(bf16x8_t v) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const bf16x2_t p = {v[2 * e], v[2 * e + 1]};
        s = __builtin_amdgcn_fdot2_f32_bf16(p, p, s, false);
    }
    return s;
}

// exact fp64 full score of row `row` for the head whose query rows are ql / qr
// (the products of two bf16 values are exact in fp64; they are added in
// dimension order from +0).  Pieces of 32 dims are loaded two pieces ahead of
// the chain (a ring of three), so the memory round trips overlap the
// arithmetic.
__device__ __forceinline__ double full_score64(const uint16_t* ql, const uint16_t* qr, const uint16_t* row) {
    constexpr int NP = D_ROW / 32;   // 18 pieces of 4 x 8 dims
    u16x8_t qv[3][4], xv[3][4];
    auto load = [&](int p, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int d = 32 * p + 8 * j;
            qv[buf][j] = *reinterpret_cast<const u16x8_t*>(d < D_LAT ? ql + d : qr + (d - D_LAT));
            xv[buf][j] = *reinterpret_cast<const u16x8_t*>(row + d);
        }
    };
    double acc = 0.0;
    auto chain = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                acc = fma((double)bf16_to_f32(qv[buf][j][e]), (double)bf16_to_f32(xv[buf][j][e]), acc);
    };
    static_assert(NP % 3 == 0, "pieces taken in threes");
    load(0, 0);
    load(1, 1);
    // a loop, not unrolled: a fully unrolled chain lets the compiler issue all
    // loads first and spill them
#pragma unroll 1
    for (int p = 0; p < NP; p += 3) {
        load(p + 2, 2);
        chain(0);
        if (p + 3 < NP) load(p + 3, 0);
        chain(1);
        if (p + 4 < NP) load(p + 4, 1);
        chain(2);
    }
    return acc;
}

// sum over the 16 lanes of each row of the wave (DPP lane permutations)
__device__ __forceinline__ float rowsum16(float v) {
    auto perm = [](float x, auto ctrl) __attribute__((always_inline)) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), decltype(ctrl)::value, 0xF, 0xF, true));
    };
    v += perm(v, std::integral_constant<int, 0xB1>{});    // quad_perm [1,0,3,2]
    v += perm(v, std::integral_constant<int, 0x4E>{});    // quad_perm [2,3,0,1]
    v += perm(v, std::integral_constant<int, 0x141>{});   // row_half_mirror
    v += perm(v, std::integral_constant<int, 0x140>{});   // row_mirror
    return v;
}

// max over the 16 lanes of each row of the wave (DPP lane permutations)
__device__ __forceinline__ float rowmax16(float v) {
    auto perm = [](float x, auto ctrl) __attribute__((always_inline)) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), decltype(ctrl)::value, 0xF, 0xF, true));
    };
    v = fmaxf(v, perm(v, std::integral_constant<int, 0xB1>{}));    // quad_perm [1,0,3,2]
    v = fmaxf(v, perm(v, std::integral_constant<int, 0x4E>{}));    // quad_perm [2,3,0,1]
    v = fmaxf(v, perm(v, std::integral_constant<int, 0x141>{}));   // row_half_mirror
    v = fmaxf(v, perm(v, std::integral_constant<int, 0x140>{}));   // row_mirror
    return v;
}

// (score desc, row asc): is (s1, u1) ahead of (s0, u0)?
__device__ __forceinline__ bool ahead(double s1, int64_t u1, double s0, int64_t u0) {
    return s1 > s0 || (s1 == s0 && u1 < u0);
}

// Block (hgb, b, sp): RM_WAVES waves, wave w taking heads 16 (RM_WAVES hgb +
// w) .. +15 of sequence b, over the sp-th of nsplit equal ranges of the list
// (each range yields the exact maximum of its own rows; row_merge_kernel takes
// the best of them, so the result is the same for any nsplit).  The block
// streams its range in tiles of RM_TILE rows through a two-stage LDS ring that
// all its waves read, so a row is fetched from memory once per block, not
// once per 16 heads.  Tile t + 1's 16-byte pieces are loaded into registers
// while tile t is scored and are written to the other stage after it; the row
// indices go out one tile earlier still.  Stage slot (r, p) holds piece
// p ^ (r mod 8) of tile row r, so the eight lanes that one 128-bit LDS read
// serves (eight rows, one piece) hit distinct bank groups.
constexpr int RM_WAVES = 8;
constexpr int VMCNT0 = 0x0F70;   // s_waitcnt operand: vmcnt 0, expcnt and lgkmcnt left alone
constexpr int RM_THREADS = 64 * RM_WAVES;
constexpr int RM_TILE = 32;                                   // rows per tile
constexpr int RM_WROWS = RM_TILE / RM_WAVES;                  // tile rows each wave loads (4)
constexpr int RM_WPIECES = RM_WROWS * (D_ROW / 8);            // their 16-byte pieces (288)
constexpr int RM_PER = (RM_WPIECES + 63) / 64;                // pieces per lane (5)

template <bool OFF32>
__global__ __launch_bounds__(RM_THREADS) void row_max_kernel(RowMaxArgs a) {
    __shared__ __align__(16) uint8_t s_x[2][RM_TILE * 2 * D_ROW];
    __shared__ int32_t s_id[2][RM_TILE];
    __shared__ float s_xn[2][RM_TILE];   // ||x_u||^2 of the stage's rows (fp32)
    __shared__ int32_t s_row[RM_WAVES][16][RM_CAND];
    __shared__ float s_ub[RM_WAVES][16][RM_CAND];
    const int HG = (a.H + 15) / 16;
    const int HGB = (HG + RM_WAVES - 1) / RM_WAVES;
    const int hgb = (int)(blockIdx.x % HGB);
    const int64_t jb = blockIdx.x / HGB;
    const int b = (int)(jb % a.B), sp = (int)(jb / a.B);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int hg = hgb * RM_WAVES + wave;
    const bool wave_on = hg < HG;   // waves past the last head group only load
    const int h0 = 16 * hg;
    const int hq = h0 + c;
    const bool hq_ok = wave_on && hq < a.H;
    const int64_t n1 = a.all_archive ? a.A : a.nrows;
    const int64_t Nall = n1 + (a.add_recent ? a.T - a.A : 0);
    const int64_t per = (Nall + a.nsplit - 1) / a.nsplit;
    const int64_t pbeg = min(Nall, (int64_t)sp * per);
    const int64_t N = min(Nall, pbeg + per);   // this block's list positions: [pbeg, N)
    const uint16_t* cb = a.cache + (int64_t)b * a.cbs;
    auto row_of = [&](int64_t p) -> int64_t {
        return p < n1 ? (a.all_archive ? p : (int64_t)a.rows[(int64_t)b * a.nrows + p]) : a.A + (p - n1);
    };
    // query fragments (A operand): head hq, dims 32 ks + 8 g; ||q_hq||^2 in fp32
    bf16x8_t qf[RM_KS];
    float qs = 0.f;
#pragma unroll
    for (int ks = 0; ks < RM_KS; ++ks) {
        const int d = 32 * ks + 8 * g;
        const int64_t hb = (int64_t)b * a.H + (hq_ok ? hq : 0);
        const uint16_t* src = d < D_LAT ? a.q_lat + hb * D_LAT + d : a.q_rope + hb * D_ROPE + (d - D_LAT);
        qf[ks] = hq_ok ? *reinterpret_cast<const bf16x8_t*>(src) : bf16x8_t{};
        qs += sumsq8(qf[ks]);
    }
    qs += __shfl_xor(qs, 16);
    qs += __shfl_xor(qs, 32);
    // per accumulator slot i: head h0 + 4 g + i; an upper bound of its ||q||
    // (the fp32 sum of 576 exact squares is within 576 * 2^-24 relative)
    // qk[i] = KE ||q|| inflated by 2^-19 (which covers the fp32 roundings of
    // qk and of the product with ||x|| below), KE = 2 (n + n/32) 2^-23
    constexpr float KE = 2.0f * (float)(D_ROW + D_ROW / 32) * 0x1p-23f;
    float qk[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float qub = sqrtf(__shfl(qs, 4 * g + i) * (1.0f + 0x1p-12f)) * (1.0f + 0x1p-20f);
        qk[i] = (KE * qub) * (1.0f + 0x1p-19f);
    }
    float M[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    // per head 4 g + i: entries in its list in byte i of ncand (the same in
    // the group's 16 lanes), and in bit i of ovf whether an entry did not fit
    // (set in the lane that had it); packed to spare registers in the loop
    uint32_t ncand = 0, ovf = 0;

    // loader: wave w moves tile rows 4 w .. 4 w + 3; its lane l takes pieces
    // q = l + 64 i (q < 288) of them, piece q mod 72 of row 4 w + q / 72 (rows
    // past the range repeat its last row; they are loaded, never scored).  A
    // row's pieces stay in one wave, so the wave also sums the row's squares
    // once for all 8 waves (the per-(row, head) band needs ||x_u||).
    // (list positions, row indices and, with OFF32, byte offsets inside the
    // sequence's cache fit 32 bits; the bases are uniform, so the loads take
    // a scalar base and a 32-bit lane offset)
    const int32_t* rb = a.rows ? a.rows + (int64_t)b * a.nrows : nullptr;
    const int32_t n1i = (int32_t)n1, Ai = (int32_t)a.A, Nm1 = (int32_t)(N - 1);
    auto load_ids = [&](int64_t t0, int32_t (&id)[RM_PER]) {
        const int32_t t0i = (int32_t)t0 + RM_WROWS * wave;
#pragma unroll
        for (int i = 0; i < RM_PER; ++i) {
            const int q = lane + 64 * i;
            if (q < RM_WPIECES) {
                const int32_t p = min(t0i + q / (D_ROW / 8), Nm1);
                int32_t v = p < n1i ? p : Ai + (p - n1i);
                if (!a.all_archive && p < n1i) v = rb[p];
                id[i] = v;
            }
        }
    };
    u32x4_t xr[RM_PER];
    const uint8_t* cbb = reinterpret_cast<const uint8_t*>(cb);
    const uint32_t rs32 = (uint32_t)(2 * a.cs);   // row stride in bytes (OFF32)
    auto load_pieces = [&](const int32_t (&id)[RM_PER]) {
#pragma unroll
        for (int i = 0; i < RM_PER; ++i) {
            const int q = lane + 64 * i;
            if (q < RM_WPIECES) {
                const int s = q % (D_ROW / 8);
                if constexpr (OFF32)
                    xr[i] = *reinterpret_cast<const u32x4_t*>(cbb + ((uint32_t)id[i] * rs32 + 16u * (uint32_t)s));
                else
                    xr[i] = *reinterpret_cast<const u32x4_t*>(cb + (int64_t)id[i] * a.cs + 8 * s);
            }
        }
    };
    auto store_pieces = [&](int st, const int32_t (&id)[RM_PER]) {
        float ns[RM_WROWS] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < RM_PER; ++i) {
            const int q = lane + 64 * i;
            if (q < RM_WPIECES) {
                const int j = q / (D_ROW / 8), s = q - (D_ROW / 8) * j;
                const int r = RM_WROWS * wave + j;
                *reinterpret_cast<u32x4_t*>(s_x[st] + r * (2 * D_ROW) + 16 * (s ^ (r & 7))) = xr[i];
                if (s == 0) s_id[st][r] = id[i];
                bf16x8_t v;
                __builtin_memcpy(&v, &xr[i], 16);
                const float ss = sumsq8(v);
#pragma unroll
                for (int jj = 0; jj < RM_WROWS; ++jj) ns[jj] += (j == jj) ? ss : 0.f;
            }
        }
        // each row's sum over the 64 lanes (16-lane rows by DPP, then across rows)
#pragma unroll
        for (int jj = 0; jj < RM_WROWS; ++jj) {
            float v = rowsum16(ns[jj]);
            v += __shfl_xor(v, 16);
            v += __shfl_xor(v, 32);
            if (lane == 0) s_xn[st][RM_WROWS * wave + jj] = v;
        }
    };

    // one 16-row half of the tile in stage st (list positions p0 ..)
    auto score_half = [&](int st, int m, int64_t p0) __attribute__((always_inline)) {
        const int rl = 16 * m + c;   // this lane's tile row
        const bool valid = p0 + c < N;
        const uint8_t* xrow = s_x[st] + rl * (2 * D_ROW);
        f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < RM_KS; ++ks) {
            const bf16x8_t xv = *reinterpret_cast<const bf16x8_t*>(xrow + 16 * ((4 * ks + g) ^ (c & 7)));
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[ks], xv, acc, 0, 0, 0);
        }
        // ||x||^2 summed by the loading wave (fp32 sums of the 576 exact
        // squares in any order are within 576 * 2^-24 relative)
        const float xs = s_xn[st][rl];
        const float xub = sqrtf(xs * (1.0f + 0x1p-12f)) * (1.0f + 0x1p-20f);
        const int32_t uc = s_id[st][rl];
        float hi[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            // e >= the band KE ||q|| ||x|| (one rounding, inside qk's slack;
            // the n 2^-120 term keeps e away from the subnormals).  The
            // rounding to nearest of acc -+ ep moves it by at most
            // 2^-24 (|acc| + ep), and ep - e >= 2^-23 (|acc| + e) exceeds that,
            // so lo <= acc - e and hi >= acc + e without directed rounding.
            const float e = fmaf(qk[i], xub, (float)D_ROW * 0x1p-120f);
            const float ep = fmaf(fabsf(acc[i]) + e, 0x1p-22f, e);
            const float lo = valid ? acc[i] - ep : -INFINITY;
            hi[i] = valid ? acc[i] + ep : -INFINITY;
            // running certified lower bound of the maximum: over the 16 rows (lanes of the group)
            M[i] = fmaxf(M[i], rowmax16(lo));
        }
        // rows whose upper bound reaches the running bound join the head's list
        // (most halves have none: one ballot per head then skips the rest)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const bool cand = hi[i] >= M[i] && valid;
            const uint64_t bal = __ballot(cand);
            if (bal == 0) continue;
            const int hl = 4 * g + i;
            const uint32_t gm = (uint32_t)(bal >> (16 * g)) & 0xFFFFu;
            int cnt = (int)((ncand >> (8 * i)) & 0xFFu);
            if (cnt + __popc(gm) > RM_CAND) {
                // prune the entries the running bound has passed (16 lanes, 4 entries each)
                int keep[4];
                int32_t kr[4];
                float ku[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int q = c + 16 * j;
                    kr[j] = s_row[wave][hl][q];
                    ku[j] = s_ub[wave][hl][q];
                    keep[j] = (q < cnt && ku[j] >= M[i]) ? 1 : 0;
                }
                __builtin_amdgcn_wave_barrier();
                int base = 0;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t km = (uint32_t)(__ballot(keep[j]) >> (16 * g)) & 0xFFFFu;
                    if (keep[j]) {
                        const int q = base + __popc(km & ((1u << c) - 1u));
                        s_row[wave][hl][q] = kr[j];
                        s_ub[wave][hl][q] = ku[j];
                    }
                    base += __popc(km);
                }
                cnt = base;
                __builtin_amdgcn_wave_barrier();
            }
            if (cand) {
                const int q = cnt + __popc(gm & ((1u << c) - 1u));
                if (q < RM_CAND) {
                    s_row[wave][hl][q] = uc;
                    s_ub[wave][hl][q] = hi[i];
                } else {
                    ovf |= 1u << i;   // more near-ties than the list holds: all rows are evaluated
                }
            }
            ncand = (ncand & ~(0xFFu << (8 * i))) | ((uint32_t)min(cnt + __popc(gm), RM_CAND) << (8 * i));
            __builtin_amdgcn_wave_barrier();
        }
    };

    const int64_t ntiles = N > pbeg ? (N - pbeg + RM_TILE - 1) / RM_TILE : 0;   // the same in every wave
    int32_t id_a[RM_PER] = {}, id_b[RM_PER] = {};
    if (ntiles > 0) {
        load_ids(pbeg, id_a);
        load_pieces(id_a);
        store_pieces(0, id_a);
    }
    if (ntiles > 1) load_ids(pbeg + RM_TILE, id_b);
    __builtin_amdgcn_s_waitcnt(VMCNT0);
    __syncthreads();
    // tile t: id_next = row indices of tile t + 1 (loaded a tile ago); the
    // indices of tile t + 2 go into id_next2.  The two index buffers swap roles
    // from tile to tile, so no register copy waits for a load.
    auto tile = [&](int64_t t, const int32_t (&id_next)[RM_PER], int32_t (&id_next2)[RM_PER])
                    __attribute__((always_inline)) {
        const int st = (int)(t & 1);
        const int64_t p0 = pbeg + RM_TILE * t;
        if (t + 1 < ntiles) load_pieces(id_next);
        if (t + 2 < ntiles) load_ids(p0 + 2 * RM_TILE, id_next2);
        if (wave_on) {
            score_half(st, 0, p0);
            score_half(st, 1, p0 + 16);
        }
        // every wave is past tile t - 1, whose stage this refills (the barrier
        // that ended it); tile t + 1 becomes visible at the barrier below
        if (t + 1 < ntiles) store_pieces(st ^ 1, id_next);
        // nothing stays in flight past a tile (the indices of tile t + 2 have
        // had the whole tile to land), so no path into the next tile leaves
        // the compiler a load it has to wait for early
        __builtin_amdgcn_s_waitcnt(VMCNT0);
        __syncthreads();
    };
    for (int64_t t = 0; t < ntiles; t += 2) {
        tile(t, id_b, id_a);
        if (t + 1 >= ntiles) break;
        tile(t + 1, id_a, id_b);
    }
    if (!wave_on) return;
    __builtin_amdgcn_wave_barrier();
    // Exact fp64 scores of the list entries whose bound reaches the final M_h.
    // The four lists of a group are taken as one sequence of (head, entry)
    // pairs dealt to its 16 lanes; a head whose list overflowed has all its
    // rows evaluated instead.
    int nl[4];
    bool over[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const bool hv = h0 + 4 * g + i < a.H;
        over[i] = hv && N > pbeg && ((uint32_t)(__ballot((ovf >> i) & 1u) >> (16 * g)) & 0xFFFFu) != 0;
        nl[i] = (!hv || over[i] || N <= pbeg) ? 0 : (int)((ncand >> (8 * i)) & 0xFFu);
    }
    double best[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    int64_t arg[4] = {-1, -1, -1, -1};
    auto offer = [&](int i, double v, int64_t u) __attribute__((always_inline)) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (k == i && ahead(v, u, best[k], arg[k])) {
                best[k] = v;
                arg[k] = u;
            }
    };
    auto head_ptrs = [&](int i, const uint16_t*& ql, const uint16_t*& qr) __attribute__((always_inline)) {
        const int h = min(h0 + 4 * g + i, a.H - 1);
        const int64_t hb = (int64_t)b * a.H + h;
        ql = a.q_lat + hb * D_LAT;
        qr = a.q_rope + hb * D_ROPE;
    };
    // the pairs whose bound reaches the final M_h, compacted per lane group
    // (into the tile ring, free now), so that the fp64 chains fill the lanes:
    // most entries of the lists fall below the final bound
    int16_t* s_pairs = reinterpret_cast<int16_t*>(&s_x[0][0]) + (wave * 4 + g) * (4 * RM_CAND);
    const int total = nl[0] + nl[1] + nl[2] + nl[3];
    int totmax = max(total, __shfl_xor(total, 16));
    totmax = max(totmax, __shfl_xor(totmax, 32));
    int npass = 0;   // the same in the group's 16 lanes
    for (int j0 = 0; j0 < totmax; j0 += 16) {
        const int j = j0 + c;
        bool pass = false;
        int code = 0;
        if (j < total) {
            const int i = j < nl[0] ? 0 : (j < nl[0] + nl[1] ? 1 : (j < nl[0] + nl[1] + nl[2] ? 2 : 3));
            const int q = j - (i > 0 ? nl[0] : 0) - (i > 1 ? nl[1] : 0) - (i > 2 ? nl[2] : 0);
            const float Mi = i == 0 ? M[0] : (i == 1 ? M[1] : (i == 2 ? M[2] : M[3]));
            pass = s_ub[wave][4 * g + i][q] >= Mi;
            code = RM_CAND * i + q;
        }
        const uint32_t gm = (uint32_t)(__ballot(pass) >> (16 * g)) & 0xFFFFu;
        if (pass) s_pairs[npass + __popc(gm & ((1u << c) - 1u))] = (int16_t)code;
        npass += __popc(gm);
    }
    __builtin_amdgcn_wave_barrier();
    for (int j = c; j < npass; j += 16) {
        const int code = s_pairs[j];
        const int i = code / RM_CAND, q = code - RM_CAND * i;
        const int64_t u = s_row[wave][4 * g + i][q];
        const uint16_t *ql, *qr;
        head_ptrs(i, ql, qr);
        offer(i, full_score64(ql, qr, cb + u * a.cs), u);
    }
#pragma unroll 1
    for (int i = 0; i < 4; ++i) {
        if (!over[i]) continue;
        const uint16_t *ql, *qr;
        head_ptrs(i, ql, qr);
        for (int64_t p = pbeg + c; p < N; p += 16) {
            const int64_t u = row_of(p);
            offer(i, full_score64(ql, qr, cb + u * a.cs), u);
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int h = h0 + 4 * g + i;
        double bv = best[i];
        int64_t ba = arg[i];
        // (max, lowest row) over the 16 lanes of the group
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
            const double ob = __shfl_xor(bv, o);
            const int64_t oa = (int64_t)__shfl_xor((long long)ba, o);
            if (oa >= 0 && ahead(ob, oa, bv, ba)) {
                bv = ob;
                ba = oa;
            }
        }
        if (c == 0 && h < a.H) {
            const int64_t hb = (int64_t)b * a.H + h;
            if (a.nsplit > 1) {
                a.part_v[hb * a.nsplit + sp] = bv;
                a.part_u[hb * a.nsplit + sp] = (int32_t)ba;
            } else {
                a.smax[hb] = bv;
                a.argmax[hb] = (int32_t)ba;
            }
        }
    }
}

// (max, lowest row) over the ranges of each (sequence, head)
__global__ __launch_bounds__(64) void row_merge_kernel(RowMaxArgs a) {
    const int64_t t = (int64_t)blockIdx.x * 64 + threadIdx.x;
    if (t >= (int64_t)a.B * a.H) return;
    double best = -INFINITY;
    int64_t arg = -1;
    for (int sp = 0; sp < a.nsplit; ++sp) {
        const double v = a.part_v[t * a.nsplit + sp];
        const int64_t u = a.part_u[t * a.nsplit + sp];
        if (u >= 0 && ahead(v, u, best, arg)) {
            best = v;
            arg = u;
        }
    }
    a.smax[t] = best;
    a.argmax[t] = (int32_t)arg;
}

hipError_t launch_row_max(const RowMaxArgs& a, hipStream_t s) {
    const int HG = (a.H + 15) / 16;
    const unsigned nblk = (unsigned)((HG + RM_WAVES - 1) / RM_WAVES * a.B * a.nsplit);
    // 32-bit byte offsets when every row of a sequence lies within 4 GiB of its first
    if ((a.T - 1) * a.cs * 2 + 2 * D_ROW <= (int64_t)UINT32_MAX)
        hipLaunchKernelGGL(row_max_kernel<true>, dim3(nblk), dim3(RM_THREADS), 0, s, a);
    else
        hipLaunchKernelGGL(row_max_kernel<false>, dim3(nblk), dim3(RM_THREADS), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.nsplit <= 1) return e;
    const int64_t n = (int64_t)a.B * a.H;
    hipLaunchKernelGGL(row_merge_kernel, dim3((unsigned)((n + 63) / 64)), dim3(64), 0, s, a);
    return hipGetLastError();
}

// one thread per (calibration query b, head h)
__global__ __launch_bounds__(64) void inflation_kernel(InflArgs a) {
    const int64_t t = (int64_t)blockIdx.x * 64 + threadIdx.x;
    if (t >= (int64_t)a.B * a.H) return;
    const int b = (int)(t / a.H);
    const int32_t u = a.argmax[t];
    bool in_s = false;
    if (u >= 0 && u < a.A && a.k > 0) {
        const int32_t* sb = a.sel + (int64_t)b * a.k;
        int64_t lo = 0, hi = a.k;   // sel is ascending
        while (lo < hi) {
            const int64_t mid = (lo + hi) / 2;
            if (sb[mid] < u) lo = mid + 1;
            else hi = mid;
        }
        in_s = lo < a.k && sb[lo] == u;
    }
    const bool hard = u >= 0 && u < a.A && !in_s;
    a.hard[t] = hard ? 1 : 0;
    double z = 0.0;
    if (hard) {
        const uint16_t* q = a.qt + t * a.n;
        const uint16_t* x = a.x + (int64_t)b * a.xbs + (int64_t)u * a.xs;
        double acc = 0.0;
        for (int d = 0; d < a.n; ++d) acc = fma((double)bf16_to_f32(q[d]), (double)bf16_to_f32(x[d]), acc);
        const float4 hs = reinterpret_cast<const float4*>(a.hsc)[t];
        const int64_t o = (int64_t)b * a.T + u;
        const double idx = acc + fma((double)hs.y, (double)a.eps[o], (double)hs.z * (double)a.gam[o]);
        const double cert = (double)hs.x * (double)a.eta[o] / sqrt((double)(D_LAT - a.r));
        const double gap = a.tier1[t] - idx;
        z = cert > 0.0 ? gap / cert : (gap > 0.0 ? INFINITY : -INFINITY);
    }
    a.zq[t] = z;
}

hipError_t launch_inflation(const InflArgs& a, hipStream_t s) {
    const int64_t n = (int64_t)a.B * a.H;
    hipLaunchKernelGGL(inflation_kernel, dim3((unsigned)((n + 63) / 64)), dim3(64), 0, s, a);
    return hipGetLastError();
}

}  // namespace vkv
