// k_page.hip -- per-page boxes of the index rows and the interval bound of a
// page (page-bound pruning; appendix "The dividend inside prior algorithms").
//
// The archived rows [0, A) of a sequence are cut into pages of `page`
// consecutive rows (the last one ragged).  The box of page j is the range of
// each index column over the page's rows, [lo_d, hi_d].  The index score is
// linear in the row for a fixed query, so the page's interval bound
//     bound_j = max_h sum_d max(qt_hd lo_d, qt_hd hi_d)
// is >= the index key of every row of the page (the page-bound equation).  The
// larger product is qt_hd hi_d for qt_hd >= 0 and qt_hd lo_d otherwise, so a
// term is one product of two bf16 values, exact in fp64; the terms are summed
// d ascending with one rounding each (v_fma_f64), the order of the fp64 index
// key.  Each term is >= the key's term and rounding is monotone, so the bound
// is >= the key bit for bit, and a page with bound < theta holds no row of the
// tier-1 set.
#include "vkv_internal.h"

namespace vkv {

constexpr int PB_PAGES = 16;    // pages per bound block
constexpr int PB_THREADS = 128; // one head per thread (H <= 128)

// Boxes: a thread takes one 8-column piece of one page and walks the page's
// rows with 16-byte loads (the n/8 threads of a page read each row as one
// contiguous run); a block covers 256 / (n/8) pages of one sequence.
// Comparisons in fp32 (exact for bf16 values); equal values have equal bits
// except for zeros, which are written as +0.
constexpr int BOX_THREADS = 256;
constexpr int BOX_UNROLL = 8;    // rows in flight per thread

__device__ __forceinline__ uint16_t box_bits(float v) {
    return v == 0.f ? (uint16_t)0 : (uint16_t)(__float_as_uint(v) >> 16);
}

__global__ __launch_bounds__(BOX_THREADS) void page_box_kernel(PageArgs a) {
    const int b = blockIdx.y;
    const int np8 = a.n / 8;                       // pieces per row
    const int ppb = BOX_THREADS / np8;             // pages per block
    const int t = threadIdx.x;
    if (t >= ppb * np8) return;
    const int64_t j = (int64_t)blockIdx.x * ppb + t / np8;
    if (j >= a.npages) return;
    const int pc = t % np8;
    const int64_t u0 = j * a.page, u1 = min(a.A, u0 + a.page);
    const uint16_t* src = a.x + (int64_t)b * a.xbs + u0 * a.xs + 8 * pc;
    float lo[8], hi[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        lo[e] = INFINITY;
        hi[e] = -INFINITY;
    }
    const int nrow = (int)(u1 - u0);
    for (int r0 = 0; r0 < nrow; r0 += BOX_UNROLL) {
        u16x8_t v[BOX_UNROLL];
#pragma unroll
        for (int i = 0; i < BOX_UNROLL; ++i)   // rows past the page re-read its last row (no effect on min/max)
            v[i] = *reinterpret_cast<const u16x8_t*>(src + (int64_t)min(r0 + i, nrow - 1) * a.xs);
#pragma unroll
        for (int i = 0; i < BOX_UNROLL; ++i)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float f = bf16_to_f32(v[i][e]);
                lo[e] = f < lo[e] ? f : lo[e];
                hi[e] = f > hi[e] ? f : hi[e];
            }
    }
    u16x8_t ol, oh;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        ol[e] = box_bits(lo[e]);
        oh[e] = box_bits(hi[e]);
    }
    uint16_t* box = a.box + ((int64_t)b * a.npages + j) * 2 * a.n;
    reinterpret_cast<u16x8_t*>(box)[pc] = ol;
    reinterpret_cast<u16x8_t*>(box + a.n)[pc] = oh;
}

__device__ __forceinline__ double bf16_f64(uint16_t b) { return (double)__uint_as_float((uint32_t)b << 16); }

// Bounds of PB_PAGES pages of sequence b: the pages' boxes are staged in LDS,
// thread h runs the chains of head h for all the pages at once (one fp64
// chain per page, d ascending), then the block takes the maximum over heads.
__global__ __launch_bounds__(PB_THREADS) void page_bound_kernel(PageArgs a) {
    extern __shared__ __align__(16) uint16_t s_box[];   // [PB_PAGES][2][n]
    __shared__ double s_best[PB_PAGES][PB_THREADS / 64];
    const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t j0 = (int64_t)blockIdx.x * PB_PAGES;
    const int np = (int)min((int64_t)PB_PAGES, a.npages - j0);
    const int n8 = a.n / 8;
    {
        const u16x8_t* src = reinterpret_cast<const u16x8_t*>(a.box + ((int64_t)b * a.npages + j0) * 2 * a.n);
        for (int p = tid; p < np * 2 * n8; p += PB_THREADS) reinterpret_cast<u16x8_t*>(s_box)[p] = src[p];
    }
    __syncthreads();
    double best[PB_PAGES];
#pragma unroll
    for (int j = 0; j < PB_PAGES; ++j) best[j] = -INFINITY;
    if (tid < a.H) {
        const u16x8_t* q = reinterpret_cast<const u16x8_t*>(a.qt + ((int64_t)b * a.H + tid) * a.n);
        double acc[PB_PAGES];
#pragma unroll
        for (int j = 0; j < PB_PAGES; ++j) acc[j] = 0.0;
        u16x8_t qn = q[0];
        for (int c = 0; c < n8; ++c) {
            const u16x8_t qv = qn;
            if (c + 1 < n8) qn = q[c + 1];   // the next piece in flight meanwhile
#pragma unroll
            for (int j = 0; j < PB_PAGES; ++j) {
                // pages past the block's last one repeat it (their chains are dropped)
                const int jj = j < np ? j : np - 1;
                const u16x8_t lo = reinterpret_cast<const u16x8_t*>(s_box + (2 * jj) * a.n)[c];
                const u16x8_t hi = reinterpret_cast<const u16x8_t*>(s_box + (2 * jj + 1) * a.n)[c];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const double qe = bf16_f64(qv[e]);
                    acc[j] = fma(qe, bf16_f64(qe >= 0.0 ? hi[e] : lo[e]), acc[j]);
                }
            }
        }
#pragma unroll
        for (int j = 0; j < PB_PAGES; ++j) best[j] = acc[j];
    }
#pragma unroll
    for (int j = 0; j < PB_PAGES; ++j) {
        double v = best[j];
        for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
        if (lane == 0) s_best[j][wave] = v;
    }
    __syncthreads();
    if (tid < np) {
        double v = s_best[tid][0];
#pragma unroll
        for (int w = 1; w < PB_THREADS / 64; ++w) v = fmax(v, s_best[tid][w]);
        a.bound[(int64_t)b * a.npages + j0 + tid] = v;
    }
}

hipError_t launch_page_box(const PageArgs& a, hipStream_t s) {
    if (a.npages == 0) return hipSuccess;
    const int ppb = BOX_THREADS / (a.n / 8);   // n <= 576: at least 3 pages per block
    hipLaunchKernelGGL(page_box_kernel, dim3((unsigned)((a.npages + ppb - 1) / ppb), a.B), dim3(BOX_THREADS), 0, s,
                       a);
    return hipGetLastError();
}

hipError_t launch_page_bound(const PageArgs& a, hipStream_t s) {
    if (a.npages == 0) return hipSuccess;
    const size_t sm = (size_t)PB_PAGES * 2 * a.n * 2;
    hipLaunchKernelGGL(page_bound_kernel, dim3((unsigned)((a.npages + PB_PAGES - 1) / PB_PAGES), a.B),
                       dim3(PB_THREADS), sm, s, a);
    return hipGetLastError();
}

}  // namespace vkv
