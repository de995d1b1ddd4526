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
// Tiles of 32 rows are double-buffered in LDS: while tile i is scored and
// accumulated, tile i+1 streams in by direct global->LDS loads
// (global_load_lds_dwordx4), row-major with piece p of tile row r at slot
// (p + r) mod 72 (conflict-free MFMA operand reads).  Once a tile has landed
// its latent half is also written transposed (for O += P V, V as the B
// operand).  P never leaves registers: the S accumulator layout of a lane (4
// rows x 1 head per 16-row tile) is exactly the A-operand layout of the PV
// product when the 32 rows of the tile are fed to the K dimension in a
// permuted order, and the transposed tile is written in that same order.
// Online softmax in the log2 domain; each split emits (unnormalised O,
// running max, running sum) and a second kernel merges the splits by their
// log-sum-exp (the appendix's kernel mapping: fetched rows are one more
// split-KV partition).
#include "vkv_internal.h"

namespace vkv {

constexpr int ATT_WAVES = ATT_HEADS / 16;     // 8
constexpr int ATT_THREADS = 64 * ATT_WAVES;  // 512
constexpr int ROW_PIECES = D_ROW / 8;        // 72 pieces of 16 B per row
constexpr int TILE_BYTES = ATT_CHUNK * D_ROW * 2;            // 36 KB
constexpr int TILE_LOADS = TILE_BYTES / 1024;                // 36 loads of 1 KB
constexpr int VT_STRIDE = 40;                // LDS stride of the transposed tile (u16), 80 B
constexpr int VT_BYTES = D_LAT * VT_STRIDE * 2;              // 40 KB

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

// Position of tile row rl on the K axis of the PV product: rows
// 16*mt + 4*g + i (held by lane group g at accumulator slot i of M-tile mt)
// go to K slot 8*g + 4*mt + i.
__device__ __forceinline__ int pv_slot(int rl) {
    return 8 * ((rl & 15) >> 2) + 4 * (rl >> 4) + (rl & 3);
}

__device__ __forceinline__ int32_t attended_row(const AttendArgs& a, int b, int64_t p) {
    if (p < a.k) return a.sel[(int64_t)b * a.k + p];
    if (p < a.k + a.W) return (int32_t)(a.A + (p - a.k));
    return a.adm[(int64_t)b * a.cap + (p - a.k - a.W)];
}

// byte offset of piece p of tile row r in a row-major stage: the slot is p
// with its low three bits XORed by (r / 2) mod 8, which spreads the 16 rows
// read by one MFMA operand load over all LDS banks (rows are 1152 B apart,
// i.e. alternate between two bank halves)
__device__ __forceinline__ int kslot(int r, int p) {
    return r * (D_ROW * 2) + 16 * (p ^ ((r >> 1) & 7));
}

__global__ __launch_bounds__(ATT_THREADS, 1) void attend_kernel(AttendArgs a) {
    extern __shared__ __align__(16) uint8_t smem[];
    uint8_t* s_k = smem;                                      // [2][TILE_BYTES]
    uint8_t* s_vt = smem + 2 * TILE_BYTES;                    // [2][D_LAT][VT_STRIDE] u16
    int32_t* s_rows = reinterpret_cast<int32_t*>(smem + 2 * TILE_BYTES + 2 * VT_BYTES);   // the split's rows

    const int sp = blockIdx.x, hg = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x;
    const int lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t nadm = (a.adm && a.cap > 0) ? min((int64_t)max(a.adm_count[b], 0), a.cap) : 0;
    const int64_t N = a.k + a.W + nadm;
    const int64_t p0 = (int64_t)sp * a.rows_per_split;
    const int64_t p1 = min(N, p0 + a.rows_per_split);
    float* po = a.part_o + ((int64_t)b * a.splits + sp) * a.H * D_LAT;
    float* pml = a.part_ml + ((int64_t)b * a.splits + sp) * a.H * 2;
    if (p0 >= p1) {
        if (tid < ATT_HEADS) {
            const int h = hg * ATT_HEADS + tid;
            if (h < a.H) {
                pml[2 * h] = -INFINITY;
                pml[2 * h + 1] = 0.f;
            }
        }
        return;
    }
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
    // direct loads of tile t into stage t & 1 (load instruction j goes to wave
    // j % 8); rows past the end of the list repeat its last row (loaded, never
    // weighted)
    auto issue = [&](int t) {
        uint8_t* st = s_k + (t & 1) * TILE_BYTES;
        for (int j = wave; j < TILE_LOADS; j += ATT_WAVES) {
            const int q = 64 * j + lane;               // destination slot
            const int r = q / ROW_PIECES, s = q % ROW_PIECES;
            const int p = s ^ ((r >> 1) & 7);
            const int i = min(ATT_CHUNK * t + r, nrow - 1);
            const uint16_t* src = cb + (int64_t)s_rows[i] * a.cs + 8 * p;
            __builtin_amdgcn_global_load_lds((gbl_void_t*)src, (lds_void_t*)(st + 1024 * j), 16, 0, 0);
        }
    };
    issue(0);

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
    float m_run = -INFINITY, l_run = 0.f;
    f32x4_t o[D_LAT / 16];
#pragma unroll
    for (int t = 0; t < D_LAT / 16; ++t) o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int t = 0; t < ntile; ++t) {
        const int cur = t & 1;
        const int nr = (int)min((int64_t)ATT_CHUNK, p1 - (p0 + (int64_t)ATT_CHUNK * t));
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's loads of tile t have landed
        __syncthreads();                                   // ... and every wave's
        if (t + 1 < ntile) issue(t + 1);
        const uint8_t* kt = s_k + cur * TILE_BYTES;
        uint16_t* vt = reinterpret_cast<uint16_t*>(s_vt + cur * VT_BYTES);
        // latent half transposed: each thread 4 pieces (row r, dims 8pc..8pc+7);
        // the 32 lanes of a half-wave take the 32 rows of one piece, so one
        // store instruction covers 32 consecutive K slots of 2 rows of V^T
#pragma unroll
        for (int jj = 0; jj < ATT_CHUNK * (D_LAT / 8) / ATT_THREADS; ++jj) {
            const int pi = tid + ATT_THREADS * jj;
            const int r = pi & (ATT_CHUNK - 1), pc = pi >> 5;
            const u16x8_t v = *reinterpret_cast<const u16x8_t*>(kt + kslot(r, pc));
            uint16_t* dst = vt + (8 * pc) * VT_STRIDE + pv_slot(r);
#pragma unroll
            for (int e = 0; e < 8; ++e) dst[e * VT_STRIDE] = v[e];
        }
        // operand of (row 16 mt + c, piece 4 ks + g): with x = (c / 2) mod 8 the
        // slot is 4 (ks ^ (x / 4)) + (g ^ (x mod 4)), so one base per ks parity
        f32x4_t sacc[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
        {
            const int x = (c >> 1) & 7;
            const uint8_t* ke = kt + c * (D_ROW * 2) + 16 * (g ^ (x & 3)) + 64 * (x >> 2);
            const uint8_t* ko = kt + c * (D_ROW * 2) + 16 * (g ^ (x & 3)) - 64 * (x >> 2);
            // operands one k-step ahead of the matrix cores
            bf16x8_t kb[2][2];
#pragma unroll
            for (int mt = 0; mt < 2; ++mt)
                kb[0][mt] = *reinterpret_cast<const bf16x8_t*>(ke + 16 * mt * (D_ROW * 2));
#pragma unroll
            for (int ks = 0; ks < D_ROW / 32; ++ks) {
                if (ks + 1 < D_ROW / 32) {
#pragma unroll
                    for (int mt = 0; mt < 2; ++mt)
                        kb[(ks + 1) & 1][mt] = *reinterpret_cast<const bf16x8_t*>(
                            (((ks + 1) & 1) ? ko : ke) + 16 * mt * (D_ROW * 2) + 64 * (ks + 1));
                }
#pragma unroll
                for (int mt = 0; mt < 2; ++mt)
                    sacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb[ks & 1][mt], qf[ks], sacc[mt], 0, 0, 0);
            }
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
        cmax = fmaxf(cmax, __shfl_xor(cmax, 16));
        cmax = fmaxf(cmax, __shfl_xor(cmax, 32));
        const float m_new = fmaxf(m_run, cmax);
        const float alpha = exp2f(m_run - m_new);
        bf16x8_t pa;
        float psum = 0.f;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = exp2f(sc[mt][i] - m_new);
                psum += p;
                pa[4 * mt + i] = (__bf16)p;
            }
        psum += __shfl_xor(psum, 16);
        psum += __shfl_xor(psum, 32);
        l_run = l_run * alpha + psum;
        m_run = m_new;
        float al[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) al[i] = __shfl(alpha, 4 * g + i);
        __syncthreads();   // transposed tile complete
        // rescale the accumulators only when some head's running max moved
        if (__ballot(alpha != 1.0f)) {
#pragma unroll
            for (int tt = 0; tt < D_LAT / 16; ++tt)
#pragma unroll
                for (int i = 0; i < 4; ++i) o[tt][i] *= al[i];
        }
        const uint16_t* vrow = &vt[c * VT_STRIDE + 8 * g];
        bf16x8_t vb[2];
        vb[0] = *reinterpret_cast<const bf16x8_t*>(vrow);
#pragma unroll
        for (int tt = 0; tt < D_LAT / 16; ++tt) {
            if (tt + 1 < D_LAT / 16) vb[(tt + 1) & 1] = *reinterpret_cast<const bf16x8_t*>(vrow + 16 * (tt + 1) * VT_STRIDE);
            o[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vb[tt & 1], o[tt], 0, 0, 0);
        }
    }
    // o[tt][i] = unnormalised output of head h0 + 4*g + i, dim 16*tt + c
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int h = h0 + 4 * g + i;
        if (h < a.H) {
#pragma unroll
            for (int tt = 0; tt < D_LAT / 16; ++tt) po[(int64_t)h * D_LAT + 16 * tt + c] = o[tt][i];
        }
    }
    if (g == 0 && hq < a.H) {
        pml[2 * hq] = m_run;
        pml[2 * hq + 1] = l_run;
    }
}

// Merge the splits of each (b, h) by log-sum-exp; bf16 output, natural-log lse.
__global__ __launch_bounds__(128) void attend_combine_kernel(AttendArgs a) {
    const int bh = blockIdx.x;
    const int b = bh / a.H, h = bh % a.H;
    const int tid = threadIdx.x;
    float M = -INFINITY;
    for (int s = 0; s < a.splits; ++s) M = fmaxf(M, a.part_ml[(((int64_t)b * a.splits + s) * a.H + h) * 2]);
    uint16_t* out = a.out + (int64_t)bh * D_LAT;
    if (M == -INFINITY) {
        for (int d = tid; d < D_LAT; d += 128) out[d] = 0;
        if (tid == 0) a.lse[bh] = -INFINITY;
        return;
    }
    float L = 0.f;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < a.splits; ++s) {
        const int64_t base = ((int64_t)b * a.splits + s) * a.H + h;
        const float ms = a.part_ml[base * 2];
        if (ms == -INFINITY) continue;
        const float w = exp2f(ms - M);
        L += w * a.part_ml[base * 2 + 1];
        const float4 v = *reinterpret_cast<const float4*>(a.part_o + base * D_LAT + 4 * tid);
        acc[0] += w * v.x;
        acc[1] += w * v.y;
        acc[2] += w * v.z;
        acc[3] += w * v.w;
    }
    const float inv = 1.0f / L;
    ushort4 r;
    r.x = f32_to_bf16_rne(acc[0] * inv);
    r.y = f32_to_bf16_rne(acc[1] * inv);
    r.z = f32_to_bf16_rne(acc[2] * inv);
    r.w = f32_to_bf16_rne(acc[3] * inv);
    *reinterpret_cast<ushort4*>(out + 4 * tid) = r;
    if (tid == 0) a.lse[bh] = (M + log2f(L)) * 0.69314718055994530942f;
}

constexpr size_t ATT_SMEM = 2 * (size_t)TILE_BYTES + 2 * (size_t)VT_BYTES + ATT_MAX_SPLIT_ROWS * sizeof(int32_t);

hipError_t launch_attend(const AttendArgs& a, hipStream_t s) {
    dim3 grid((unsigned)a.splits, (unsigned)((a.H + ATT_HEADS - 1) / ATT_HEADS), (unsigned)a.B);
    hipError_t e0 = hipFuncSetAttribute(reinterpret_cast<const void*>(attend_kernel),
                                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)ATT_SMEM);
    if (e0 != hipSuccess) return e0;
    hipLaunchKernelGGL(attend_kernel, grid, dim3(ATT_THREADS), ATT_SMEM, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attend_combine_kernel, dim3((unsigned)(a.B * a.H)), dim3(128), 0, s, a);
    return hipGetLastError();
}

}  // namespace vkv
