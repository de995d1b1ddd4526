// k_digest.hip -- index build (the compression event's tier-2 index, Sec. 4.2).
//
// Archived row u keeps (r_u, P c_u, eta_u); with the stored sketch rounded to
// bf16 the certificate needs two more row scalars (eps_u, gamma_u).  For each
// row: y_j = sum_i P[j,i] c_u[i] in fp64 with i ascending, d_j = RNE_bf16(y_j)
// in one rounding, then the upper bounds
//   eta_u >= sqrt(c^T (I - P^T P) c),  eps_u >= ||d - P c||,  gamma_u >= ||P c||
// evaluated in a fixed fp64 order and rounded toward +inf.  Not on the
// per-step path.  A block owns 32 rows; the basis is held
// transposed in LDS, 64 columns at a time.
#include "vkv_internal.h"

namespace vkv {

constexpr int DG_THREADS = 256;

__global__ __launch_bounds__(DG_THREADS) void digest_kernel(DigestArgs a, int rows_per_block) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t(*s_pt)[66] = reinterpret_cast<uint16_t(*)[66]>(smem);                       // [512][66]
    double(*s_c)[D_LAT] = reinterpret_cast<double(*)[D_LAT]>(smem + D_LAT * 66 * 2);     // [4][512]
    double(*s_y)[64] = reinterpret_cast<double(*)[64]>(smem + D_LAT * 66 * 2 + 4 * D_LAT * 8);  // [R][64]

    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int64_t u0 = (int64_t)blockIdx.x * rows_per_block;
    const int nrows = (int)min((int64_t)rows_per_block, a.T - u0);
    if (nrows <= 0) return;
    const uint16_t* cb = a.cache + (int64_t)b * a.cbs;
    uint16_t* ib = a.index ? a.index + (int64_t)b * a.ibs : nullptr;
    const int off = a.with_rope ? D_ROPE : 0;

    // running sums of the row owners (thread rho < nrows), in j order
    double Ny = 0.0, Ne = 0.0;

    const int ntile = (a.r + 63) / 64;
    for (int jt = 0; jt < ntile; ++jt) {
        const int j0 = 64 * jt;
        const int jn = min(64, a.r - j0);
        __syncthreads();
        for (int idx = tid; idx < jn * D_LAT; idx += DG_THREADS) {
            const int jl = idx / D_LAT, i = idx % D_LAT;
            s_pt[i][jl] = a.P[(int64_t)(j0 + jl) * D_LAT + i];
        }
        for (int rg = 0; rg < nrows; rg += 4) {
            __syncthreads();
            for (int idx = tid; idx < 4 * D_LAT; idx += DG_THREADS) {
                const int rl = idx / D_LAT, i = idx % D_LAT;
                const int rr = rg + rl;
                s_c[rl][i] = (rr < nrows) ? (double)bf16_to_f32(cb[(u0 + rr) * a.cs + i]) : 0.0;
            }
            __syncthreads();
            const int rl = tid >> 6, jl = tid & 63;
            const int rr = rg + rl;
            if (rr < nrows && jl < jn) {
                double acc = 0.0;
                for (int i = 0; i < D_LAT; ++i) acc = fma((double)bf16_to_f32(s_pt[i][jl]), s_c[rl][i], acc);
                s_y[rr][jl] = acc;
                if (ib) ib[(u0 + rr) * a.is + off + j0 + jl] = f64_to_bf16_rne(acc);
            }
        }
        __syncthreads();
        if (tid < nrows) {
            for (int jl = 0; jl < jn; ++jl) {
                const double y = s_y[tid][jl];
                Ny = fma(y, y, Ny);
            }
            for (int jl = 0; jl < jn; ++jl) {
                const double y = s_y[tid][jl];
                const double t = (double)bf16_to_f32(f64_to_bf16_rne(y)) - y;
                Ne = fma(t, t, Ne);
            }
        }
    }
    // branch copy (the exact summand of every future logit)
    if (ib && a.with_rope) {
        for (int idx = tid; idx < nrows * (D_ROPE / 8); idx += DG_THREADS) {
            const int rr = idx / (D_ROPE / 8), p = idx % (D_ROPE / 8);
            *reinterpret_cast<u16x8_t*>(ib + (u0 + rr) * a.is + 8 * p) =
                *reinterpret_cast<const u16x8_t*>(cb + (u0 + rr) * a.cs + D_LAT + 8 * p);
        }
    }
    if (a.eta && tid < nrows) {
        const uint16_t* c = cb + (u0 + tid) * a.cs;
        double Nc = 0.0;
        for (int i = 0; i < D_LAT; ++i) {
            const double v = (double)bf16_to_f32(c[i]);
            Nc = fma(v, v, Nc);
        }
        const double G = CERT_G;
        const double Dm = G * (double)ru_sqrt_f32((double)a.r * Nc);
        const double sy = (double)ru_sqrt_f32(Ny);
        const double X = ((Nc - Ny) + G * (Nc + Ny)) + (2.0 * Dm) * sy;
        const int64_t o = (int64_t)b * a.T + u0 + tid;
        a.eta[o] = ru_sqrt_f32((X > 0.0 ? X : 0.0) * (1.0 + G));
        a.eps[o] = ru_f32((double)ru_sqrt_f32(Ne) * (1.0 + G) + Dm);
        a.gam[o] = ru_f32(sy * (1.0 + G) + Dm);
    }
}

static size_t digest_smem(int rows_per_block) {
    return (size_t)D_LAT * 66 * 2 + 4 * D_LAT * 8 + (size_t)rows_per_block * 64 * 8;
}

hipError_t launch_digest(const DigestArgs& a, hipStream_t s) {
    if (a.T <= 0) return hipSuccess;
    const int rpb = 32;
    const size_t sm = digest_smem(rpb);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(digest_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)((a.T + rpb - 1) / rpb), (unsigned)a.B);
    hipLaunchKernelGGL(digest_kernel, grid, dim3(DG_THREADS), sm, s, a, rpb);
    return hipGetLastError();
}

// Gershgorin row sums of P P^T: rowsum[j] = sum_k |sum_i P[j,i] P[k,i]|, with
// flag[j] = 1 if any fp64 addition on the way rounded (TwoSum error != 0).
// bf16 products are exact in fp64, so flag 0 means rowsum[j] is exact.
__device__ __forceinline__ double two_sum_add(double a, double b, int* inexact) {
    const double s = a + b;
    const double bp = s - a;
    const double err = (a - (s - bp)) + (b - bp);
    if (err != 0.0) *inexact = 1;
    return s;
}

__global__ __launch_bounds__(256) void gram_rows_kernel(const uint16_t* P, int r, double* rowsum, double* flag) {
    __shared__ double s_g[512];
    __shared__ int s_f[512];
    const int j = blockIdx.x;
    const int tid = threadIdx.x;
    for (int k = tid; k < r; k += 256) {
        double gk = 0.0;
        int inexact = 0;
        for (int i = 0; i < D_LAT; ++i) {
            const double p = (double)bf16_to_f32(P[(int64_t)j * D_LAT + i]) * (double)bf16_to_f32(P[(int64_t)k * D_LAT + i]);
            gk = two_sum_add(gk, p, &inexact);
        }
        s_g[k] = gk;
        s_f[k] = inexact;
    }
    __syncthreads();
    if (tid == 0) {
        double acc = 0.0;
        int inexact = 0;
        for (int k = 0; k < r; ++k) {
            acc = two_sum_add(acc, fabs(s_g[k]), &inexact);
            inexact |= s_f[k];
        }
        rowsum[j] = acc;
        flag[j] = inexact ? 1.0 : 0.0;
    }
}

hipError_t launch_gram_rows(const uint16_t* P, int r, double* rowsum, hipStream_t s) {
    if (r <= 0) return hipSuccess;
    hipLaunchKernelGGL(gram_rows_kernel, dim3(r), dim3(256), 0, s, P, r, rowsum, rowsum + 512);
    return hipGetLastError();
}

}  // namespace vkv
