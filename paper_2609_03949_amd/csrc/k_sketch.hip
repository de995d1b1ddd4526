// k_sketch.hip -- the data-driven sketch basis V_r of the index (Sec. 4.2,
// the index entry: the rank-r sketch of the content uses V_r drawn from the
// context's own prefix queries).
//
// V_r spans the dominant r-dimensional eigenspace of the prefix content
// queries' second moment C = sum_i q_i q_i^T (512 x 512).  The index score
// (V_r^T q).(V_r^T c) = q^T V_r V_r^T c and the residual norm
// ||(I - V_r V_r^T) c|| depend on the subspace only, so any orthonormal basis
// of it serves; the basis is found by subspace (orthogonal) iteration:
//   V_0 = orth(C R) with R a fixed +-1 pattern, V_{t+1} = orth(C V_t),
// orth = Cholesky QR applied twice (W = V L^T with L L^T = W^T W), all fp64.
// The error shrinks as (lambda_{r+1} / lambda_r)^t.  The products are tiled
// fp64 kernels; the r x r factorisation runs in one block.  The basis is handed to
// vkv_digest_build as P = RNE_bf16(s V_r^T), s = 1 - 2^-6, which keeps the
// rounded basis contractive (checked there).  Not on the per-step path: it is
// part of the compression event.
#include "vkv_internal.h"

namespace vkv {

constexpr int SK_T = 64;        // output tile of the fp64 products (64 x 64 or 64 x 32)
constexpr int SK_K = 32;        // inner-dimension chunk staged in LDS
constexpr double SK_SCALE = 1.0 - 0x1p-6;

// C[a][b] = sum_i q[i][a] q[i][b] over the m queries (bf16 products exact in fp64).
// Block (ta, tb) owns the 64 x 64 tile; 256 threads hold 4 x 4 outputs each.
__global__ __launch_bounds__(256) void cov_kernel(const uint16_t* q, int64_t m, double* C) {
    __shared__ double sa[SK_K][SK_T + 1], sb[SK_K][SK_T + 1];
    const int ta = blockIdx.x, tb = blockIdx.y, tid = threadIdx.x;
    const int ra = (tid / 16) * 4, rb = (tid % 16) * 4;
    double acc[4][4] = {};
    for (int64_t i0 = 0; i0 < m; i0 += SK_K) {
        for (int e = tid; e < SK_K * SK_T; e += 256) {
            const int i = e / SK_T, j = e % SK_T;
            const bool in = i0 + i < m;
            sa[i][j] = in ? (double)bf16_to_f32(q[(i0 + i) * D_LAT + ta * SK_T + j]) : 0.0;
            sb[i][j] = in ? (double)bf16_to_f32(q[(i0 + i) * D_LAT + tb * SK_T + j]) : 0.0;
        }
        __syncthreads();
        for (int i = 0; i < SK_K; ++i)
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 4; ++y) acc[x][y] = fma(sa[i][ra + x], sb[i][rb + y], acc[x][y]);
        __syncthreads();
    }
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) C[(int64_t)(ta * SK_T + ra + x) * D_LAT + tb * SK_T + rb + y] = acc[x][y];
}

__global__ __launch_bounds__(64) void sk_zero_kernel(int* p) {
    if (threadIdx.x == 0) p[0] = 0;
}

// The fixed +-1 start pattern R[i][j]: the top bit of MurmurHash3's 32-bit
// finaliser (fmix32) of i * 512 + j plus a constant.  (A hash whose low bits
// are weakly mixed gives a pattern of low rank; this one is well conditioned.)
__device__ __forceinline__ double start_pattern(int i, int j) {
    uint32_t h = (uint32_t)(i * D_LAT + j) + 0x5BD1E995u;
    h ^= h >> 16;
    h *= 0x85EBCA6Bu;
    h ^= h >> 13;
    h *= 0xC2B2AE35u;
    h ^= h >> 16;
    return (h >> 31) ? 1.0 : -1.0;
}

// Out[a][c] = sum_k A(a, k) B(k, c) for a < M, c < N, k < K (fp64, k ascending
// per output), A(a, k) = A[a*sa0 + k*sa1], B(k, c) = B[k*sb0 + c*sb1]; Out is
// row-major with N columns.  B == nullptr stands for the start pattern.
// Block (ta, tc) owns 64 rows x 32 columns; 256 threads hold 2 x 4 outputs.
struct Mat {
    const double* p;
    int64_t s0, s1;
};

__global__ __launch_bounds__(256) void gemm64_kernel(Mat A, Mat B, int M, int N, int K, double* Out) {
    __shared__ double sa[SK_T][SK_K + 1], sb[SK_K][32 + 1];
    const int ta = blockIdx.x, tc = blockIdx.y, tid = threadIdx.x;
    const int ra = (tid / 8) * 2, rc = (tid % 8) * 4;
    double acc[2][4] = {};
    for (int k0 = 0; k0 < K; k0 += SK_K) {
        for (int e = tid; e < SK_T * SK_K; e += 256) {
            const int i = e / SK_K, k = e % SK_K, row = ta * SK_T + i;
            sa[i][k] = (row < M && k0 + k < K) ? A.p[row * A.s0 + (k0 + k) * A.s1] : 0.0;
        }
        for (int e = tid; e < SK_K * 32; e += 256) {
            const int k = e / 32, j = e % 32, col = tc * 32 + j;
            const bool in = col < N && k0 + k < K;
            sb[k][j] = in ? (B.p ? B.p[(k0 + k) * B.s0 + col * B.s1] : start_pattern(k0 + k, col)) : 0.0;
        }
        __syncthreads();
        for (int k = 0; k < SK_K; ++k)
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 4; ++y) acc[x][y] = fma(sa[ra + x][k], sb[k][rc + y], acc[x][y]);
        __syncthreads();
    }
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) {
            const int row = ta * SK_T + ra + x, col = tc * 32 + rc + y;
            if (row < M && col < N) Out[(int64_t)row * N + col] = acc[x][y];
        }
}

// One block: G (r x r, symmetric positive definite) -> its Cholesky factor L
// in place (lower triangle, right-looking), then Li = L^{-1} (lower
// triangular; one thread per column, forward substitution).  A pivot that is
// not finite or not above SK_PIV_REL times its column's original diagonal sets
// *bad: the columns are numerically dependent (Cholesky QR needs the condition
// number of the columns below about 1e7).
constexpr double SK_PIV_REL = 1e-15;

__global__ __launch_bounds__(256) void chol_inv_kernel(double* G, int r, double* Li, int* bad) {
    const int tid = threadIdx.x;
    __shared__ double s_piv;
    __shared__ int s_bad;
    if (tid == 0) s_bad = 0;
    // the original diagonal, kept on Li's diagonal until Li is formed
    for (int j = tid; j < r; j += 256) Li[(int64_t)j * r + j] = G[(int64_t)j * r + j];
    __syncthreads();
    for (int j = 0; j < r; ++j) {
        if (tid == 0) {
            double d = G[(int64_t)j * r + j];
            if (!(d > SK_PIV_REL * Li[(int64_t)j * r + j]) || !(d < INFINITY)) {
                s_bad = 1;
                d = 1.0;
            }
            s_piv = sqrt(d);
            G[(int64_t)j * r + j] = s_piv;
        }
        __syncthreads();
        for (int i = j + 1 + tid; i < r; i += 256) G[(int64_t)i * r + j] /= s_piv;
        __syncthreads();
        const int n = r - j - 1;
        for (int e = tid; e < n * n; e += 256) {
            const int i = j + 1 + e / n, l = j + 1 + e % n;
            if (l <= i) G[(int64_t)i * r + l] -= G[(int64_t)i * r + j] * G[(int64_t)l * r + j];
        }
        __syncthreads();
    }
    for (int c = tid; c < r; c += 256) {
        for (int i = 0; i < c; ++i) Li[(int64_t)i * r + c] = 0.0;
        Li[(int64_t)c * r + c] = 1.0 / G[(int64_t)c * r + c];
        for (int i = c + 1; i < r; ++i) {
            double s = 0.0;
            for (int k = c; k < i; ++k) s = fma(G[(int64_t)i * r + k], Li[(int64_t)k * r + c], s);
            Li[(int64_t)i * r + c] = -s / G[(int64_t)i * r + i];
        }
    }
    if (tid == 0 && s_bad) *bad = 1;
}

// P[j][i] = RNE_bf16(s V[i][j]); quot[j] = v_j^T C v_j (the Rayleigh quotient
// of column j).  Block j; each thread takes rows a of C v_j, then a block sum.
__global__ __launch_bounds__(256) void basis_out_kernel(const double* V, const double* C, int r, uint16_t* P,
                                                        double* quot) {
    const int j = blockIdx.x, tid = threadIdx.x;
    __shared__ double red[256];
    for (int i = tid; i < D_LAT; i += 256) P[(int64_t)j * D_LAT + i] = f64_to_bf16_rne(SK_SCALE * V[(int64_t)i * r + j]);
    double s = 0.0;
    for (int a = tid; a < D_LAT; a += 256) {
        double t = 0.0;
        for (int b2 = 0; b2 < D_LAT; ++b2) t = fma(C[(int64_t)a * D_LAT + b2], V[(int64_t)b2 * r + j], t);
        s = fma(V[(int64_t)a * r + j], t, s);
    }
    red[tid] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (tid < w) red[tid] += red[tid + w];
        __syncthreads();
    }
    if (tid == 0) quot[j] = red[0];
}

// energy[0] = sum_j quot[j] = trace(V^T C V) (j ascending), energy[1] = trace(C) (a ascending)
__global__ __launch_bounds__(64) void energy_kernel(const double* quot, const double* C, int r, double* energy) {
    if (threadIdx.x != 0) return;
    double e0 = 0.0, e1 = 0.0;
    for (int j = 0; j < r; ++j) e0 += quot[j];
    for (int a = 0; a < D_LAT; ++a) e1 += C[(int64_t)a * D_LAT + a];
    energy[0] = e0;
    energy[1] = e1;
}

size_t sketch_workspace_bytes(int r) {
    return (size_t)D_LAT * D_LAT * 8 + 2 * (size_t)D_LAT * r * 8 + 2 * (size_t)r * r * 8 + 256;
}

static hipError_t gemm(Mat A, Mat B, int M, int N, int K, double* Out, hipStream_t s) {
    const dim3 g((unsigned)((M + SK_T - 1) / SK_T), (unsigned)((N + 31) / 32));
    hipLaunchKernelGGL(gemm64_kernel, g, dim3(256), 0, s, A, B, M, N, K, Out);
    return hipGetLastError();
}

hipError_t launch_sketch(const uint16_t* q, int64_t m, int r, int iters, void* ws, uint16_t* P, double* energy,
                         hipStream_t s) {
    double* C = reinterpret_cast<double*>(ws);
    double* X = C + (size_t)D_LAT * D_LAT;     // the basis (512 x r)
    double* Y = X + (size_t)D_LAT * r;         // its image / the second orthonormalisation
    double* G = Y + (size_t)D_LAT * r;         // Gram matrix, then its Cholesky factor
    double* Li = G + (size_t)r * r;            // inverse factor
    int* bad = reinterpret_cast<int*>(Li + (size_t)r * r);
    hipLaunchKernelGGL(sk_zero_kernel, dim3(1), dim3(64), 0, s, bad);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(cov_kernel, dim3(D_LAT / SK_T, D_LAT / SK_T), dim3(256), 0, s, q, m, C);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // orth(src -> dst): G = src^T src, L L^T = G, dst = src L^{-T}
    auto orth = [&](const double* src, double* dst) -> hipError_t {
        hipError_t e2 = gemm(Mat{src, 1, r}, Mat{src, r, 1}, r, r, D_LAT, G, s);
        if (e2 != hipSuccess) return e2;
        hipLaunchKernelGGL(chol_inv_kernel, dim3(1), dim3(256), 0, s, G, r, Li, bad);
        if ((e2 = hipGetLastError()) != hipSuccess) return e2;
        return gemm(Mat{src, r, 1}, Mat{Li, 1, r}, D_LAT, r, r, dst, s);
    };
    for (int t = 0; t <= iters; ++t) {
        // Y = C X (the start pattern on the first round), then X = orth(orth(Y))
        if ((e = gemm(Mat{C, D_LAT, 1}, Mat{t == 0 ? nullptr : X, r, 1}, D_LAT, r, D_LAT, Y, s)) != hipSuccess)
            return e;
        if ((e = orth(Y, X)) != hipSuccess) return e;
        if ((e = orth(X, Y)) != hipSuccess) return e;
        double* tmp = X;
        X = Y;
        Y = tmp;
    }
    hipLaunchKernelGGL(basis_out_kernel, dim3((unsigned)r), dim3(256), 0, s, X, C, r, P, Li);
    if ((e = hipGetLastError()) != hipSuccess || !energy) return e;
    hipLaunchKernelGGL(energy_kernel, dim3(1), dim3(64), 0, s, Li, C, r, energy);
    return hipGetLastError();
}

}  // namespace vkv
