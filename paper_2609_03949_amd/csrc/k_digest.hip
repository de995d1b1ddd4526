// k_digest.hip -- index build (the compression event's tier-2 index, Sec. 4.2).
//
// Archived row u keeps (r_u, P c_u, eta_u); with the stored sketch rounded to
// bf16 the certificate needs two more row scalars (eps_u, gamma_u).  For each
// row: y_j = sum_i P[j,i] c_u[i] in fp64 with i ascending, d_j = RNE_bf16(y_j)
// in one rounding, then the upper bounds
//   eta_u >= sqrt(c^T (I - P^T P) c),  eps_u >= ||d - P c||,  gamma_u >= ||P c||
// evaluated in a fixed fp64 order and rounded toward +inf.  Not on the
// per-step path.
//
// The projection runs on the fp64 matrix cores: v_mfma_f64_16x16x4f64 adds its
// 4 products (k = 0..3) to the accumulator one after another, each with a
// single rounding, so 128 of them with i ascending give the sequential fp64
// sum bit for bit (bf16 products are exact in fp64).  A block owns DG_ROWS
// consecutive rows of one sequence and takes the basis in chunks of 64 rows
// (one 16-row tile per wave): each chunk is staged once in LDS, and the
// block's rows stream past it in two streams of 16-row tiles, so that each
// SIMD runs two independent chains (double-buffered: each stream's next tile
// is loaded into registers during the current tile's chain).
// Rows and basis rows sit in LDS rows padded to DG_ROW bytes, so the operand
// reads (16 rows, one 16-bit element each) fall into distinct banks.  The
// row sums over j (||y||^2, ||d - y||^2) continue chunk after chunk in j
// order; ||c||^2 runs on the vector unit of wave 0 between its matrix steps.
#include <type_traits>

#include "vkv_internal.h"

namespace vkv {

constexpr int DG_THREADS = 512;   // two streams of 4 waves: one basis tile per wave, two row tiles at a time
constexpr int DG_ROW = 1040;       // LDS bytes per staged row of 512 bf16
constexpr int DG_CHUNK = 64;       // basis rows per chunk: 16 per wave of a stream
constexpr int DG_ROWS = 256;       // cache rows per block (16 tiles of 16)

typedef __attribute__((address_space(3))) void dg_lds_t;
typedef __attribute__((address_space(1))) void dg_gbl_t;

__global__ __launch_bounds__(DG_THREADS) void digest_kernel(DigestArgs a) {
    __shared__ __align__(16) uint8_t s_p[DG_CHUNK * DG_ROW];        // a chunk of basis rows
    __shared__ __align__(16) uint8_t s_c[2][2][16 * DG_ROW];        // per stream, two tiles of cache rows
    __shared__ double s_y[2][16][DG_CHUNK];                         // per stream, y of its tile and the chunk
    __shared__ double s_acc[DG_ROWS][2];                            // running ||y||^2, ||d - y||^2
    __shared__ double s_nc[DG_ROWS];                                // ||c||^2

    const int b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int st = wave >> 2, jw = wave & 3;   // row stream, basis tile of the chunk
    const int stid = tid & 255;                // thread index within the stream
    const int64_t u0 = (int64_t)blockIdx.x * DG_ROWS;
    const int nrows = (int)min((int64_t)DG_ROWS, a.T - u0);
    if (nrows <= 0) return;
    const int ntile = (nrows + 15) / 16;
    const int niter = (ntile + 1) / 2;   // stream st takes tiles 2 it + st
    const uint16_t* cb = a.cache + (int64_t)b * a.cbs;
    uint16_t* ib = a.index ? a.index + (int64_t)b * a.ibs : nullptr;
    const int off = a.with_rope ? D_ROPE : 0;
    const bool cert = a.eta != nullptr;
    for (int i = tid; i < DG_ROWS; i += DG_THREADS) s_acc[i][0] = s_acc[i][1] = 0.0;

    // this stream's tile of iteration 0 into its buffer 0 (4 rows per wave,
    // one 1 KB load each); rows past T are zero
    auto stage_first = [&]() {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int rl = 4 * jw + q, rr = 16 * st + rl;
            uint8_t* dst = s_c[st][0] + rl * DG_ROW;
            if (rr < nrows)
                __builtin_amdgcn_global_load_lds((dg_gbl_t*)(cb + (u0 + rr) * a.cs + 8 * lane), (dg_lds_t*)dst, 16, 0, 0);
            else
                *reinterpret_cast<u32x4_t*>(dst + 16 * lane) = u32x4_t{0u, 0u, 0u, 0u};
        }
    };
    const int nchunk = a.r > 0 ? (a.r + DG_CHUNK - 1) / DG_CHUNK : 1;
    for (int ch = 0; ch < nchunk; ++ch) {
        const int j0 = ch * DG_CHUNK;
        const int jn = a.r > 0 ? min(DG_CHUNK, a.r - j0) : 0;
        __syncthreads();   // the previous chunk's reads of s_p and s_c are done
        for (int row = wave; row < jn; row += DG_THREADS / 64)
            __builtin_amdgcn_global_load_lds((dg_gbl_t*)(a.P + (int64_t)(j0 + row) * D_LAT + 8 * lane),
                                             (dg_lds_t*)(s_p + row * DG_ROW), 16, 0, 0);
        stage_first();
        const bool tile = 16 * jw < jn;
        const bool nc = ch == 0 && jw == 0 && cert;
        // operand rows: A = cache row (lane mod 16) of the tile, B = basis row
        // 16 jw + (lane mod 16) of the chunk; element k = lane / 16 of each step
        const uint16_t* pb = reinterpret_cast<const uint16_t*>(s_p + (16 * jw + (lane & 15)) * DG_ROW) + (lane >> 4);
        for (int it = 0; it < niter; ++it) {
            const int t = 2 * it + st;
            const bool have = t < ntile;
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();   // tile t (and the chunk) landed; buffer (it+1)&1 and s_y are free
            // the stream's next tile into registers now, into LDS after the
            // chain: no direct load into LDS is in flight while the chain reads
            // it, so the compiler's LDS wait counts stay exact
            u32x4_t nx[4];
            const int tn = t + 2;
            const bool more = tn < ntile;
            if (more) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int rr = 16 * tn + 4 * jw + q;
                    nx[q] = rr < nrows ? *reinterpret_cast<const u32x4_t*>(cb + (u0 + rr) * a.cs + 8 * lane)
                                       : u32x4_t{0u, 0u, 0u, 0u};
                }
            }
            const uint8_t* tb = s_c[st][it & 1];
            const uint16_t* ca = reinterpret_cast<const uint16_t*>(tb + (lane & 15) * DG_ROW) + (lane >> 4);
            const uint16_t* cn = reinterpret_cast<const uint16_t*>(tb + (lane & 15) * DG_ROW);
            f64x4_t acc = f64x4_t{0.0, 0.0, 0.0, 0.0};
            double anc = 0.0;
            if (have) {
                if (tile && nc) acc = mfma_f64_rowdot512<true>(ca, pb, cn, anc);
                else if (tile) acc = mfma_f64_rowdot512<false>(ca, pb, cn, anc);
                else if (nc) {
                    for (int i = 0; i < D_LAT; ++i) {
                        const double x = bf16_bits_f64(cn[i]);
                        anc = fma(x, x, anc);
                    }
                }
            }
            if (more) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    *reinterpret_cast<u32x4_t*>(s_c[st][(it + 1) & 1] + (4 * jw + q) * DG_ROW + 16 * lane) = nx[q];
            }
            if (have && nc && lane < 16 && 16 * t + lane < nrows) s_nc[16 * t + lane] = anc;
            if (have && tile) {
                // acc[i] = y of tile row 4 i + lane / 16, basis row j0 + 16 jw + lane mod 16
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int rl = 4 * i + (lane >> 4), jl = 16 * jw + (lane & 15);
                    const double y = acc[i];
                    s_y[st][rl][jl] = y;
                    const int rr = 16 * t + rl;
                    if (ib && rr < nrows) ib[(u0 + rr) * a.is + off + j0 + jl] = f64_to_bf16_rne(y);
                }
            }
            if (have && ch == 0 && ib && a.with_rope) {
                // branch copy (the exact summand of every future logit): 16 rows x 128 B
                const int rl = stid >> 4, p = stid & 15;
                const int rr = 16 * t + rl;
                if (p < D_ROPE / 8 && rr < nrows)
                    *reinterpret_cast<u16x8_t*>(ib + (u0 + rr) * a.is + 8 * p) =
                        *reinterpret_cast<const u16x8_t*>(cb + (u0 + rr) * a.cs + D_LAT + 8 * p);
            }
            if (!cert) continue;
            __syncthreads();   // s_y complete
            if (have && jw == 0 && lane < 32) {
                // lane rl + 16 m continues sum m of tile row rl over this chunk's j, ascending
                const int rl = lane & 15, m = lane >> 4, rr = 16 * t + rl;
                double sacc = rr < nrows ? s_acc[rr][m] : 0.0;
                for (int jl = 0; jl < jn; ++jl) {
                    const double y = s_y[st][rl][jl];
                    const double v = m ? (double)bf16_to_f32(f64_to_bf16_rne(y)) - y : y;
                    sacc = fma(v, v, sacc);
                }
                if (rr < nrows) s_acc[rr][m] = sacc;
            }
        }
    }
    if (!cert) return;
    __syncthreads();
    for (int rr = tid; rr < nrows; rr += DG_THREADS) {
        const double Nc = s_nc[rr], Ny = s_acc[rr][0], Ne = s_acc[rr][1];
        const double G = CERT_G;
        const double Dm = G * (double)ru_sqrt_f32((double)a.r * Nc);
        const double sy = (double)ru_sqrt_f32(Ny);
        const double X = ((Nc - Ny) + G * (Nc + Ny)) + (2.0 * Dm) * sy;
        const int64_t o = (int64_t)b * a.T + u0 + rr;
        a.eta[o] = ru_sqrt_f32((X > 0.0 ? X : 0.0) * (1.0 + G));
        a.eps[o] = ru_f32((double)ru_sqrt_f32(Ne) * (1.0 + G) + Dm);
        a.gam[o] = ru_f32(sy * (1.0 + G) + Dm);
    }
}

hipError_t launch_digest(const DigestArgs& a, hipStream_t s) {
    if (a.T <= 0) return hipSuccess;
    dim3 grid((unsigned)((a.T + DG_ROWS - 1) / DG_ROWS), (unsigned)a.B);
    hipLaunchKernelGGL(digest_kernel, grid, dim3(DG_THREADS), 0, s, a);
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
