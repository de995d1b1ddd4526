// k_attend.hip -- split-KV gather-attend over full 576-wide rows (gfx950).
//
// For sequence b the attended multiset is  S_b ++ [A, T) ++ admitted_b  (the
// kept/recent tier plus the fetched rows, which join the softmax as exact
// copies: Lemma (Exchangeability)).  Scores use the absorbed query over all
// 576 dims and the value is the 512-dim latent (Sec. 3, Eq. (setup)):
//   s_h(u) = scale * (q_lat_h . c_u + q_rope_h . r_u),   o_h = sum_u softmax(s_h)_u c_u
//
// Work split: workgroup = (split of the row list, group of 64 heads, b);
// 4 waves x 16 heads.  Per tile of 32 rows the gathered rows are staged in
// LDS twice: row-major (for S = K Q^T, K = rows as the MFMA A operand) and
// transposed (for O += P V, V as the B operand).  P never leaves registers:
// the S accumulator layout of a lane (4 rows x 1 head per 16-row tile) is
// exactly the A-operand layout of the PV product when the 32 rows of the
// tile are fed to the K dimension in a permuted order, and the transposed V
// tile is written in that same order.  Online softmax in the log2 domain;
// each split emits (unnormalised O, running max, running sum) and a second
// kernel merges the splits by their log-sum-exp (the appendix's kernel
// mapping: fetched rows are one more split-KV partition).
#include "vkv_internal.h"

namespace vkv {

constexpr int ATT_THREADS = 256;
constexpr int KROW = D_ROW + 8;       // LDS row stride of the row-major tile (u16), 1168 B
constexpr int VT_STRIDE = 40;         // LDS stride of the transposed tile (u16), 80 B

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

__global__ __launch_bounds__(ATT_THREADS, 2) void attend_kernel(AttendArgs a) {
    __shared__ __align__(16) uint16_t s_k[ATT_CHUNK][KROW];
    __shared__ __align__(16) uint16_t s_vt[D_LAT][VT_STRIDE];
    __shared__ int32_t s_rows[ATT_CHUNK];

    const int sp = blockIdx.x, hg = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, g = lane >> 4, c = lane & 15;
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
    const int h0 = hg * ATT_HEADS + wave * 16;
    const int hq = h0 + c;
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
    const uint16_t* cb = a.cache + (int64_t)b * a.cbs;

    for (int64_t c0 = p0; c0 < p1; c0 += ATT_CHUNK) {
        const int nr = (int)min((int64_t)ATT_CHUNK, p1 - c0);
        __syncthreads();
        if (tid < ATT_CHUNK) s_rows[tid] = (tid < nr) ? attended_row(a, b, c0 + tid) : 0;
        __syncthreads();
        // gather: 32 rows x 72 pieces of 16 B = 9 pieces per thread, loaded in
        // three batches of three (each batch in flight together; the register
        // budget does not allow all nine)
        constexpr int NPIECE = ATT_CHUNK * (D_ROW / 8) / ATT_THREADS;
        constexpr int NBATCH = 3;
        static_assert(NPIECE * ATT_THREADS == ATT_CHUNK * (D_ROW / 8), "tile must split evenly");
        static_assert(NPIECE % NBATCH == 0, "batches must split evenly");
#pragma unroll 1
        for (int j0 = 0; j0 < NPIECE; j0 += NBATCH) {
            u16x8_t v[NBATCH];
#pragma unroll
            for (int j = 0; j < NBATCH; ++j) {
                const int p = tid + ATT_THREADS * (j0 + j);
                const int rl = p / (D_ROW / 8), pc = p % (D_ROW / 8);
                v[j] = (rl < nr) ? *reinterpret_cast<const u16x8_t*>(cb + (int64_t)s_rows[rl] * a.cs + 8 * pc)
                                 : u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
            }
#pragma unroll
            for (int j = 0; j < NBATCH; ++j) {
                const int p = tid + ATT_THREADS * (j0 + j);
                const int rl = p / (D_ROW / 8), pc = p % (D_ROW / 8);
                *reinterpret_cast<u16x8_t*>(&s_k[rl][8 * pc]) = v[j];
                if (pc < D_LAT / 8) {
                    // staggered element order spreads the 64 lanes over the LDS banks
                    const int pos = pv_slot(rl);
                    const int rot = pc + (pc >> 3);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int e2 = (e + rot) & 7;
                        s_vt[8 * pc + e2][pos] = v[j][e2];
                    }
                }
            }
        }
        __syncthreads();
        // S^T[row][head] for the 32 rows (two 16-row M tiles) and 16 heads
        f32x4_t sacc[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int ks = 0; ks < D_ROW / 32; ++ks)
#pragma unroll
            for (int mt = 0; mt < 2; ++mt) {
                const bf16x8_t ka = *reinterpret_cast<const bf16x8_t*>(&s_k[16 * mt + c][32 * ks + 8 * g]);
                sacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[ks], sacc[mt], 0, 0, 0);
            }
        // sacc[mt][i] = score of row 16*mt + 4*g + i for head hq
        float t[2][4];
        float cmax = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rl = 16 * mt + 4 * g + i;
                const float v = (rl < nr) ? sacc[mt][i] * a.scale_log2 : -INFINITY;
                t[mt][i] = v;
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
                const float p = exp2f(t[mt][i] - m_new);
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
#pragma unroll
        for (int tt = 0; tt < D_LAT / 16; ++tt) {
#pragma unroll
            for (int i = 0; i < 4; ++i) o[tt][i] *= al[i];
            const bf16x8_t vb = *reinterpret_cast<const bf16x8_t*>(&s_vt[16 * tt + c][8 * g]);
            o[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vb, o[tt], 0, 0, 0);
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

hipError_t launch_attend(const AttendArgs& a, hipStream_t s) {
    dim3 grid((unsigned)a.splits, (unsigned)((a.H + ATT_HEADS - 1) / ATT_HEADS), (unsigned)a.B);
    hipLaunchKernelGGL(attend_kernel, grid, dim3(ATT_THREADS), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attend_combine_kernel, dim3((unsigned)(a.B * a.H)), dim3(128), 0, s, a);
    return hipGetLastError();
}

}  // namespace vkv
