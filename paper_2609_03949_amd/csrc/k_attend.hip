// k_attend.hip -- split-KV gather-attend over full 576-wide rows (gfx950).
//
// For sequence b the attended multiset is  S_b ++ [A, T) ++ admitted_b  (the
// kept/recent tier plus the fetched rows, which join the softmax as exact
// copies: Lemma (Exchangeability)).  Scores use the absorbed query over all
// 576 dims and the value is the 512-dim latent (Sec. 3, Eq. (setup)):
//   s_h(u) = scale * (q_lat_h . c_u + q_rope_h . r_u),   o_h = sum_u softmax(s_h)_u c_u
//
// Work split: workgroup = (split of the row list, group of 128 heads, b);
// 8 waves x 16 heads, so every gathered row serves all heads of the group.
// Tiles of 32 rows stream through a ring of four LDS stages by direct
// global->LDS loads (global_load_lds_dwordx4): tiles go in groups of two, the
// next group is loaded while the current one is processed, and one workgroup
// barrier per group suffices.  Stage layout: row-major, piece p (16 B)
// of tile row r at slot 72 r + (p ^ f(r)); f spreads both operand reads below
// over all LDS banks.  S^T = K Q^T reads K rows as the A operand; O += P V
// reads V = the latent half of the same stage with the transposing LDS load
// (ds_read_b64_tr_b16), so no transposed copy is written.  P never leaves
// registers: the S accumulator layout of a lane (4 rows x 1 head per 16-row
// tile) is the A-operand layout of the PV product when the 32 rows of the tile
// are fed to the K dimension in a permuted order, which the V reads follow.
// Online softmax in the log2 domain against a reference maximum that moves
// only when a score exceeds it by more than a factor 2^8 (so P <= 256 in bf16 and the
// accumulators are rarely rescaled); each split emits (unnormalised O,
// reference max, running sum) and a second kernel merges the splits by their
// log-sum-exp (the appendix's kernel mapping: fetched rows are one more
// split-KV partition).
#include <type_traits>

#include "vkv_internal.h"

namespace vkv {

constexpr int ATT_WAVES = ATT_HEADS / 16;     // 8
constexpr int ATT_THREADS = 64 * ATT_WAVES;  // 512
constexpr int ROW_PIECES = D_ROW / 8;        // 72 pieces of 16 B per row
constexpr int TILE_BYTES = ATT_CHUNK * D_ROW * 2;            // 36 KB
constexpr int TILE_LOADS = TILE_BYTES / 1024;                // 36 loads of 1 KB
constexpr int ATT_GROUP = 2;                 // tiles per workgroup barrier
constexpr float ATT_SLACK = 8.0f;            // lag allowed to the softmax reference maximum (log2 units)
constexpr int ATT_STAGES = 2 * ATT_GROUP;    // ring depth: the group in use and the next in flight
constexpr int ROW_BYTES = D_ROW * 2;                         // 1152

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;
typedef short i16x4_t __attribute__((ext_vector_type(4)));

// rows attended by sequence b: kept, window, admitted (up to the capacity)
__device__ __forceinline__ int64_t attended_count(const AttendArgs& a, int b) {
    const int64_t nadm = (a.adm && a.cap > 0) ? min((int64_t)max(a.adm_count[b], 0), a.cap) : 0;
    return a.k + a.W + nadm;
}

// list positions [p0, p1) of split sp (empty past the end of the list)
__device__ __forceinline__ void split_range(const AttendArgs& a, int sp, int64_t N, int64_t& p0, int64_t& p1) {
    const int64_t base_end = (int64_t)a.base_splits * a.rows_per_split;
    if (sp < a.base_splits) {
        p0 = (int64_t)sp * a.rows_per_split;
        p1 = min(N, p0 + a.rows_per_split);
    } else {
        p0 = base_end + (int64_t)(sp - a.base_splits) * a.rows_per_adm;
        p1 = min(N, p0 + a.rows_per_adm);
    }
    p1 = max(p1, p0);
}

// the number of splits that hold rows of a list of N rows (32-bit: lists,
// splits and their rows are far below 2^31)
__device__ __forceinline__ int live_splits(const AttendArgs& a, int64_t N) {
    const int n = (int)N, rps = (int)a.rows_per_split, rpa = (int)a.rows_per_adm;
    const int base_end = a.base_splits * rps;
    if (n <= base_end) return (n + rps - 1) / rps;
    return a.base_splits + (n - base_end + rpa - 1) / rpa;
}

__device__ __forceinline__ int32_t attended_row(const AttendArgs& a, int b, int64_t p) {
    if (p < a.k) return a.sel[(int64_t)b * a.k + p];
    if (p < a.k + a.W) return (int32_t)(a.A + (p - a.k));
    return a.adm[(int64_t)b * a.cap + (p - a.k - a.W)];
}

// XOR applied to the piece index of tile row r (low three bits only, so each
// aligned group of 8 pieces maps onto itself): f(r) = r mod 8.  Slot (r, p)
// is 72 r + (p ^ f(r)) and 72 is a multiple of 8, so modulo 8 slots (one
// 128-byte sweep of the banks) it is p ^ f(r).  The 128-bit K operand reads
// are served eight lanes (eight rows of one piece) at a time, and r mod 8
// gives those eight rows eight distinct slots; the transposing V reads (four
// rows x two adjacent pieces per 16 lanes) stay distinct as well.  Measured with
// SQ_LDS_BANK_CONFLICT: no conflicts on either read (the previous mapping,
// which paired rows 2i and 2i + 1, doubled the K reads' LDS cycles).
__device__ __forceinline__ int piece_xor(int r) { return r & 7; }

__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Compile-time loop: f(std::integral_constant<int, I>) for I = 0 .. N-1.
template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<I + 1, N>(f);
    }
}

// op-reduction of x over the four 16-lane groups (lanes c, c+16, c+32, c+48),
// result in all of them: two cross-lane swaps, no LDS traffic
template <typename Op>
__device__ __forceinline__ float allreduce_groups(float x, Op op) {
    const uint32_t u = __float_as_uint(x);
    const auto r32 = __builtin_amdgcn_permlane32_swap(u, u, false, false);   // lane l ^ 32
    const float y = op(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
    const uint32_t v = __float_as_uint(y);
    const auto r16 = __builtin_amdgcn_permlane16_swap(v, v, false, false);   // lane l ^ 16
    return op(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
}

// Operand reads of the tile stages, issued as explicit LDS instructions: the
// compiler sees no LDS read of a stage, so it never makes them wait for the
// direct loads still in flight into the other stages, and the lgkmcnt waits
// before each use are explicit (lds_wait: at most N of this wave's LDS
// operations outstanding; LDS operations complete in order).  The kernel
// issues no scalar memory loads inside the tile loop, so lgkmcnt counts LDS
// operations only there.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
template <int OFF>
__device__ __forceinline__ bf16x8_t lds_read128(uint32_t addr) {
    bf16x8_t v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
    return v;
}
// transposing read: within each 16-lane group, lane j supplies the address of
// 4 consecutive 16-bit elements D[j][0..3], and lane i receives D[4e + i/4][i % 4]
// for e = 0..3
template <int OFF>
__device__ __forceinline__ i16x4_t lds_read_tr16(uint32_t addr) {
    i16x4_t v;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
    return v;
}
template <int N, typename T0, typename T1>
__device__ __forceinline__ void lds_wait(T0& x, T1& y) {
    asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(x), "+v"(y) : "n"(N));
}

__global__ __launch_bounds__(ATT_THREADS, 1) void attend_kernel(AttendArgs a) {
    __shared__ __align__(16) uint8_t s_k[ATT_STAGES * TILE_BYTES];   // the ring of tile stages
    __shared__ int32_t s_rows[ATT_MAX_SPLIT_ROWS];                    // the split's rows

    const int HG = (a.H + ATT_HEADS - 1) / ATT_HEADS;
    // Workgroup ids: first every base split (split, then head group, then
    // sequence), then the admitted-row workgroups j = 0, 1, ... of every
    // (head group, sequence).  Workgroups are dispatched in id order, so the
    // base splits and the first admitted workgroup of each sequence (the only
    // one with rows when few are admitted) go out before the idle ones.
    int first, hg, b;
    {
        const int64_t L = blockIdx.x;
        const int64_t nbase = (int64_t)a.B * HG * a.base_splits;
        if (L < nbase) {
            first = (int)(L % a.base_splits);
            const int64_t r = L / a.base_splits;
            hg = (int)(r % HG);
            b = (int)(r / HG);
        } else {
            const int64_t L2 = L - nbase, per = (int64_t)a.B * HG;
            first = a.base_splits + (int)(L2 / per);
            const int64_t r = L2 % per;
            hg = (int)(r % HG);
            b = (int)(r / HG);
        }
    }
    const int tid = threadIdx.x;
    const int lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t N = attended_count(a, b);

    // one split: list positions [p0, p1), p0 < p1 (splits without rows are
    // never run: the combine reads only the splits that hold rows)
    auto run_split = [&](const int sp, const int64_t p0, const int64_t p1) __attribute__((always_inline)) {
    uint16_t* po = a.part_o + (((int64_t)b * a.splits + sp) * HG + hg) * (ATT_HEADS * D_LAT);
    float* pml = a.part_ml + ((int64_t)b * a.splits + sp) * a.H * 2;
    const int ntile = (int)((p1 - p0 + ATT_CHUNK - 1) / ATT_CHUNK);
    const int h0 = hg * ATT_HEADS + wave * 16;
    const int hq = h0 + c;
    const uint16_t* cb = a.cache + (int64_t)b * a.cbs;

    // the split's row list into LDS (all loads in flight), once
    const int nrow = (int)(p1 - p0);
    {
        constexpr int PER = ATT_MAX_SPLIT_ROWS / ATT_THREADS;
        int32_t rv[PER];
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int i = tid + ATT_THREADS * j;
            rv[j] = (i < nrow) ? attended_row(a, b, p0 + i) : 0;
        }
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int i = tid + ATT_THREADS * j;
            if (i < nrow) s_rows[i] = rv[j];
        }
    }
    __syncthreads();
    // Direct loads of tile t into stage t mod 3: load instruction j (1 KB,
    // slots 64 j .. 64 j + 63) belongs to wave j mod 8, so waves 0-3 issue 5
    // per tile and waves 4-7 issue 4.  Slot q holds piece (q mod 72) ^ f(r) of
    // tile row r = q / 72.  Rows past the end of the list repeat its last row
    // (loaded, never weighted).
    constexpr int MAXJ = (TILE_LOADS + ATT_WAVES - 1) / ATT_WAVES;   // 5
    const int nj = (TILE_LOADS - wave + ATT_WAVES - 1) / ATT_WAVES;  // 5 or 4
    auto issue = [&](int t, uint8_t* st) {
        // the per-load slot arithmetic is redone each time (an opaque copy of
        // the lane index keeps the compiler from holding it across the loop)
        int ln = lane;
        asm volatile("" : "+v"(ln));
        int row[MAXJ], off[MAXJ];
#pragma unroll
        for (int i = 0; i < MAXJ; ++i) {   // all row lookups first (in bounds for every i)
            const int q = 64 * (wave + ATT_WAVES * i) + ln;
            const int r = q / ROW_PIECES;
            row[i] = s_rows[min(ATT_CHUNK * t + r, nrow - 1)];
            off[i] = 8 * ((q - ROW_PIECES * r) ^ piece_xor(r));
        }
        static_assert(MAXJ == 5, "row lookups tied below");
        asm volatile("" : "+v"(row[0]), "+v"(row[1]), "+v"(row[2]), "+v"(row[3]), "+v"(row[4]));   // one LDS round trip
#pragma unroll
        for (int i = 0; i < MAXJ; ++i) {
            if (i < nj) {
                const uint16_t* src = cb + (int64_t)row[i] * a.cs + off[i];
                __builtin_amdgcn_global_load_lds((gbl_void_t*)src, (lds_void_t*)(st + 1024 * (wave + ATT_WAVES * i)),
                                                 16, 0, 0);
            }
        }
    };
#pragma unroll
    for (int t = 0; t < ATT_GROUP; ++t)
        if (t < ntile) issue(t, s_k + t * TILE_BYTES);

    // Q fragments (B operand of S^T = K Q^T): head hq, dims 32*ks + 8*g .. +8
    bf16x8_t qf[D_ROW / 32];
#pragma unroll
    for (int ks = 0; ks < D_ROW / 32; ++ks) {
        const int d = 32 * ks + 8 * g;
        if (hq < a.H) {
            const uint16_t* src = (d < D_LAT) ? a.q_lat + ((int64_t)b * a.H + hq) * D_LAT + d
                                              : a.q_rope + ((int64_t)b * a.H + hq) * D_ROPE + (d - D_LAT);
            qf[ks] = *reinterpret_cast<const bf16x8_t*>(src);
        } else {
            qf[ks] = bf16x8_t{};
        }
    }
    // consume the query loads here, so no wait for them lands inside the tile loop
#pragma unroll
    for (int ks = 0; ks < D_ROW / 32; ++ks) asm volatile("" : "+v"(qf[ks]));
    float m_run = -INFINITY, l_run = 0.f;
    f32x4_t o[D_LAT / 16];
#pragma unroll
    for (int t = 0; t < D_LAT / 16; ++t) o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // K operand of (row 16 mt + c, piece 4 ks + g): slot low bits (4 (ks & 1) + g) ^ f(c),
    // so one byte offset per ks parity, plus 128 B per pair of k-steps.
    // V operand (transposing reads): lane j = 4e + q of group g reads tile row
    // 4g + e (and 16 + 4g + e), dims 16 tt + 4q .. +3, i.e. piece 2tt + q/2,
    // half q mod 2; the piece's low bits (2 (tt mod 4) + q/2) ^ f(row) give one
    // offset per tt mod 4, plus 128 B per four tt (f(16 + r) = f(r)).
    // Both are recomputed per tile from an opaque copy of the lane index, so the
    // compiler keeps no per-stage copies of them across the loop.
    struct Offs {
        int k_even, k_odd, v_base, v_h, v_f;
    };
    auto offsets = [&]() {
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int cc = ln & 15, gg = ln >> 4, fc = piece_xor(cc);
        const int e = cc >> 2, q = ln & 3;
        return Offs{cc * ROW_BYTES + 16 * (gg ^ fc), cc * ROW_BYTES + 16 * ((4 + gg) ^ fc),
                    (4 * gg + e) * ROW_BYTES + 8 * (q & 1), q >> 1, piece_xor(4 * gg + e)};
    };

    const uint32_t k_lds = lds_addr(s_k);
    int stage = 0;   // t mod ATT_STAGES
    for (int t = 0; t < ntile; ++t) {
        const int nr = (int)min((int64_t)ATT_CHUNK, p1 - (p0 + (int64_t)ATT_CHUNK * t));
        if (t % ATT_GROUP == 0) {
            // this wave's loads of the group t .. t+ATT_GROUP-1 have landed (nothing
            // else is in flight) ...
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            // ... and every wave's; every wave is also done with the previous group,
            // whose stages the next group reuses
            wg_barrier();
#pragma unroll
            for (int u = 0; u < ATT_GROUP; ++u) {
                const int tn = t + ATT_GROUP + u;
                if (tn < ntile) issue(tn, s_k + (tn % ATT_STAGES) * TILE_BYTES);
            }
        }
        const uint32_t kt = k_lds + (uint32_t)(stage * TILE_BYTES);
        stage = stage == ATT_STAGES - 1 ? 0 : stage + 1;
        const Offs of = offsets();
        f32x4_t sacc[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
        {
            // K operands SD k-steps ahead of the matrix cores
            constexpr int SD = 2, KSN = D_ROW / 32;
            const uint32_t ke = kt + of.k_even, ko = kt + of.k_odd;
            bf16x8_t kb[SD + 1][2];
            auto kload = [&](auto kc) {
                constexpr int ks = decltype(kc)::value;
                constexpr int off = 128 * (ks >> 1);
                const uint32_t base = (ks & 1) ? ko : ke;
                kb[ks % (SD + 1)][0] = lds_read128<off>(base);
                kb[ks % (SD + 1)][1] = lds_read128<off + 16 * ROW_BYTES>(base);
            };
            static_for<0, SD>(kload);
            static_for<0, KSN>([&](auto kc) {
                constexpr int ks = decltype(kc)::value;
                if constexpr (ks + SD < KSN) kload(std::integral_constant<int, ks + SD>{});
                constexpr int after = 2 * ((ks + SD < KSN) ? SD : (KSN - 1 - ks));
                lds_wait<after>(kb[ks % (SD + 1)][0], kb[ks % (SD + 1)][1]);
#pragma unroll
                for (int mt = 0; mt < 2; ++mt)
                    sacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb[ks % (SD + 1)][mt], qf[ks], sacc[mt], 0, 0, 0);
            });
        }
        // sacc[mt][i] = score of row 16*mt + 4*g + i for head hq
        float sc[2][4];
        float cmax = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rl = 16 * mt + 4 * g + i;
                const float v = (rl < nr) ? sacc[mt][i] * a.scale_log2 : -INFINITY;
                sc[mt][i] = v;
                cmax = fmaxf(cmax, v);
            }
        cmax = allreduce_groups(cmax, [](float x, float y) { return fmaxf(x, y); });
        // the reference maximum moves only when a score exceeds it by more than
        // ATT_SLACK (log2 units), so P <= 2^ATT_SLACK and most tiles rescale nothing
        const bool move = cmax > m_run + ATT_SLACK;
        const float m_new = move ? cmax : m_run;
        const float alpha = move ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;
        bf16x8_t pa;
        float psum = 0.f;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = __builtin_amdgcn_exp2f(sc[mt][i] - m_new);
                psum += p;
                pa[4 * mt + i] = (__bf16)p;
            }
        psum = allreduce_groups(psum, [](float x, float y) { return x + y; });
        l_run = l_run * alpha + psum;
        m_run = m_new;
        // the softmax's cross-lane reads complete before the PV reads are issued
        asm volatile("" : "+v"(l_run), "+v"(pa));
        // rescale the accumulators only when some head's reference maximum moved
        if (__ballot(move)) {
            float al[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) al[i] = __shfl(alpha, 4 * g + i);
#pragma unroll
            for (int tt = 0; tt < D_LAT / 16; ++tt)
#pragma unroll
                for (int i = 0; i < 4; ++i) o[tt][i] *= al[i];
        }
        // O += P V: B operand of dims 16 tt .. +15 = tile rows (4g + e, 16 + 4g + e)
        // at dim 16 tt + c, read VD steps ahead; dims in the order tt = 4 a + be
        // (be outer), so one address per be is live
        constexpr int VD = 3, TTN = D_LAT / 16;
        i16x4_t vv[VD + 1][2];
        uint32_t voff[4];
        auto vload = [&](auto ic) {
            constexpr int i = decltype(ic)::value;
            constexpr int tt = 4 * (i & 7) + (i >> 3);
            if constexpr ((i & 7) == 0) voff[i >> 3] = kt + of.v_base + 16 * ((2 * (tt & 3) + of.v_h) ^ of.v_f);
            vv[i % (VD + 1)][0] = lds_read_tr16<128 * (tt >> 2)>(voff[i >> 3]);
            vv[i % (VD + 1)][1] = lds_read_tr16<128 * (tt >> 2) + 16 * ROW_BYTES>(voff[i >> 3]);
        };
        static_for<0, VD>(vload);
        static_for<0, TTN>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            constexpr int tt = 4 * (i & 7) + (i >> 3);
            if constexpr (i + VD < TTN) vload(std::integral_constant<int, i + VD>{});
            constexpr int after = 2 * ((i + VD < TTN) ? VD : (TTN - 1 - i));
            lds_wait<after>(vv[i % (VD + 1)][0], vv[i % (VD + 1)][1]);
            bf16x8_t vop;
            __builtin_memcpy(&vop, vv[i % (VD + 1)], 16);
            o[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vop, o[tt], 0, 0, 0);
        });
    }
    // o[tt][i] = unnormalised output of head h0 + 4*g + i, dim 16*tt + c; the
    // partial is stored as bf16 (RNE) in that register order (one 512 B store
    // per tt and wave)
    uint16_t* pw = po + (int64_t)wave * (D_LAT / 16) * 64 * 4;
#pragma unroll
    for (int tt = 0; tt < D_LAT / 16; ++tt) {
        typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
        const bf16x4_t v = {(__bf16)o[tt][0], (__bf16)o[tt][1], (__bf16)o[tt][2], (__bf16)o[tt][3]};
        *reinterpret_cast<bf16x4_t*>(pw + (tt * 64 + lane) * 4) = v;
    }
    if (g == 0 && hq < a.H) {
        pml[2 * hq] = m_run;
        pml[2 * hq + 1] = l_run;
    }
    };

    // A base split's workgroup runs that split.  The admitted rows' splits:
    // workgroup base_splits + j takes splits base_splits + j, + adm_blocks, ...
    // until one holds no rows (they fill in order), so a mostly unused
    // capacity costs a few idle workgroups and a full one is shared by all of
    // them.  (One loop, so the split's code is generated once.)
    const int stride = first < a.base_splits ? 0 : a.adm_blocks;
    for (int sp = first; sp < a.splits; sp += stride) {
        int64_t p0, p1;
        split_range(a, sp, N, p0, p1);
        if (p0 >= p1) break;
        run_split(sp, p0, p1);
        if (stride == 0) break;
        __syncthreads();   // the row list and the ring are free before the next split refills them
    }
}

// Merge the splits of four heads by log-sum-exp (partials bf16, sums fp32);
// bf16 output, natural-log lse.
// Block = (b, head group, wave, lane group g) of the attention kernel: heads
// hb + i (i = 0..3) with hb = 128 hg + 16 wave + 4 g; thread j covers dims
// 4j .. 4j+3 (tt = j / 4, lanes 16 g + 4 (j mod 4) .. +3 of the partials).
// Splits are taken COMB_SPLITS at a time with all their loads in flight
// together (one memory round trip per batch); the running maximum and the
// accumulators are rescaled when a batch raises the maximum.
constexpr int COMB_SPLITS = 8;

__global__ __launch_bounds__(128) void attend_combine_kernel(AttendArgs a) {
    const int HG = (a.H + ATT_HEADS - 1) / ATT_HEADS;
    const int q = blockIdx.x % 32, hg = (blockIdx.x / 32) % HG, b = blockIdx.x / (32 * HG);
    const int wave = q >> 2, g = q & 3;
    const int hb = hg * ATT_HEADS + 16 * wave + 4 * g;
    if (hb >= a.H) return;
    const int j = threadIdx.x, tt = j >> 2, c0 = 4 * (j & 3);
    float M[4], L[4] = {0.f, 0.f, 0.f, 0.f};
    float acc[4][4] = {};
#pragma unroll
    for (int i = 0; i < 4; ++i) M[i] = -INFINITY;
    // only the splits that hold rows are read (none for an empty list)
    const int nlive = min(a.splits, live_splits(a, attended_count(a, b)));
    for (int s0 = 0; s0 < nlive; s0 += COMB_SPLITS) {
        float ms[COMB_SPLITS][4], ls[COMB_SPLITS][4];
        u32x4_t raw[COMB_SPLITS][2];
#pragma unroll
        for (int u = 0; u < COMB_SPLITS; ++u) {
            const int s = s0 + u;
            const bool live = s < nlive;
            const float* ml = a.part_ml + (((int64_t)b * a.splits + (live ? s : s0)) * a.H) * 2;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const bool hv = live && hb + i < a.H;
                ms[u][i] = hv ? ml[2 * (hb + i)] : -INFINITY;
                ls[u][i] = hv ? ml[2 * (hb + i) + 1] : 0.f;
            }
            // every split below nlive holds rows, so its partial was written;
            // past it the batch re-reads split s0 (weight 0), so that all loads
            // go out together, unconditionally (one round trip per batch)
            const uint16_t* src = a.part_o + (((int64_t)b * a.splits + (live ? s : s0)) * HG + hg) * (ATT_HEADS * D_LAT) +
                                  (int64_t)wave * (D_LAT / 16) * 64 * 4 + (tt * 64 + 16 * g + c0) * 4;
            raw[u][0] = *reinterpret_cast<const u32x4_t*>(src);       // lanes c0, c0+1
            raw[u][1] = *reinterpret_cast<const u32x4_t*>(src + 8);   // lanes c0+2, c0+3
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float mb = M[i];
#pragma unroll
            for (int u = 0; u < COMB_SPLITS; ++u) mb = fmaxf(mb, ms[u][i]);
            if (mb != M[i]) {   // raised (so mb is finite): rescale what is accumulated
                const float sc = (M[i] == -INFINITY) ? 0.f : exp2f(M[i] - mb);
                L[i] *= sc;
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) acc[cc][i] *= sc;
                M[i] = mb;
            }
        }
#pragma unroll
        for (int u = 0; u < COMB_SPLITS; ++u) {
            float w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                w[i] = (ms[u][i] == -INFINITY) ? 0.f : exp2f(ms[u][i] - M[i]);
                L[i] += w[i] * ls[u][i];
            }
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) {
                const u32x4_t& rw = raw[u][cc >> 1];
                const uint32_t w01 = rw[2 * (cc & 1)], w23 = rw[2 * (cc & 1) + 1];
                const float v[4] = {__uint_as_float(w01 << 16), __uint_as_float(w01 & 0xFFFF0000u),
                                    __uint_as_float(w23 << 16), __uint_as_float(w23 & 0xFFFF0000u)};
                // a split without rows never wrote its partial: weight 0 must not touch it
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[cc][i] += (w[i] > 0.f) ? w[i] * v[i] : 0.f;
            }
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int h = hb + i;
        if (h >= a.H) continue;
        uint16_t* out = a.out + ((int64_t)b * a.H + h) * D_LAT + 4 * j;
        ushort4 r{0, 0, 0, 0};
        if (M[i] != -INFINITY) {
            const float inv = 1.0f / L[i];
            r.x = f32_to_bf16_rne(acc[0][i] * inv);
            r.y = f32_to_bf16_rne(acc[1][i] * inv);
            r.z = f32_to_bf16_rne(acc[2][i] * inv);
            r.w = f32_to_bf16_rne(acc[3][i] * inv);
        }
        *reinterpret_cast<ushort4*>(out) = r;
        if (j == 0)
            a.lse[(int64_t)b * a.H + h] =
                (M[i] == -INFINITY) ? -INFINITY : (M[i] + log2f(L[i])) * 0.69314718055994530942f;
    }
}

hipError_t launch_attend(const AttendArgs& a, hipStream_t s) {
    const int64_t nwg = (int64_t)(a.base_splits + a.adm_blocks) * ((a.H + ATT_HEADS - 1) / ATT_HEADS) * a.B;
    hipLaunchKernelGGL(attend_kernel, dim3((unsigned)nwg), dim3(ATT_THREADS), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned hgs = (unsigned)((a.H + ATT_HEADS - 1) / ATT_HEADS);
    hipLaunchKernelGGL(attend_combine_kernel, dim3((unsigned)a.B * hgs * 32u), dim3(128), 0, s, a);
    return hipGetLastError();
}

}  // namespace vkv
