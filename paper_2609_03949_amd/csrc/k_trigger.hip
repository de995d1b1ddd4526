// k_trigger.hip -- the tier-1 maximum logit and the calibration statistic of
// the calibrated trigger (Sec. 4.2: Eq. (trigger), the z paragraph; Sec. 5.2).
//
// row_max_kernel: per sequence b and head h, the maximum over a row list of
// the exact full score s_h(u) = q_lat_h . c_u + q_rope_h . r_u (Sec. 3,
// Eq. (setup); the fp64 sum over the 576 dims, latent then branch, from +0)
// and the row attaining it (ties: the lower row index).  Over the tier-1
// rows it is the trigger threshold s*_h; over the whole context it is the
// causal argmax row of a calibration query.  One wave per (sequence, 16
// heads) streams the list: bf16 MFMA scores in fp32 with a per-(row, head)
// certified band e = 2 (n + n/32) 2^-23 ||q_h|| ||x_u|| (n = 576, the
// scan's error model), a running certified lower bound M_h of the maximum,
// and in LDS the rows whose upper bound reaches M_h.  Only those get the
// fp64 chain; the true maximum row always does.
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
__device__ __forceinline__ double full_score64(const uint16_t* ql, const uint16_t* qr, const uint16_t* row) {
    double acc = 0.0;
#pragma unroll 1
    for (int p0 = 0; p0 < D_ROW / 8; p0 += 8) {
        u16x8_t qv[8], xv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int d = 8 * (p0 + j);
            qv[j] = *reinterpret_cast<const u16x8_t*>(d < D_LAT ? ql + d : qr + (d - D_LAT));
            xv[j] = *reinterpret_cast<const u16x8_t*>(row + d);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc = fma((double)bf16_to_f32(qv[j][e]), (double)bf16_to_f32(xv[j][e]), acc);
    }
    return acc;
}

// (score desc, row asc): is (s1, u1) ahead of (s0, u0)?
__device__ __forceinline__ bool ahead(double s1, int64_t u1, double s0, int64_t u0) {
    return s1 > s0 || (s1 == s0 && u1 < u0);
}

// s_waitcnt operand that waits for vmcnt 0 and leaves expcnt and lgkmcnt alone
constexpr int VMCNT0 = 0x0F70;

// Block (hg, b, sp): heads 16 hg .. of sequence b over the sp-th of nsplit
// equal ranges of the list (the ranges are exact maxima of their own rows;
// row_merge_kernel takes the best of them, so the result is the same for any
// nsplit).  The blocks of one (b, sp) read the same rows, so when the number
// of (b, sp) items is a multiple of 8 they are given linear ids that are equal
// mod 8: workgroups are dealt to the 8 XCDs round-robin by linear id, so all
// head groups of a range share one XCD's L2.
__global__ __launch_bounds__(64) void row_max_kernel(RowMaxArgs a) {
    __shared__ int32_t s_row[16][RM_CAND];
    __shared__ float s_ub[16][RM_CAND];
    __shared__ int s_cnt[16];
    __shared__ int s_over[16];
    const int HG = (a.H + 15) / 16;
    const int64_t items = (int64_t)a.B * a.nsplit;
    int hg, b, sp;
    {
        const int64_t L = blockIdx.x;
        int64_t j;
        if (items % 8 == 0) {
            const int64_t rest = L / 8;
            hg = (int)(rest % HG);
            j = (L % 8) + 8 * (rest / HG);
        } else {
            hg = (int)(L % HG);
            j = L / HG;
        }
        b = (int)(j % a.B);
        sp = (int)(j / a.B);
    }
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    const int h0 = 16 * hg;
    const int hq = h0 + c;
    const bool hq_ok = hq < a.H;
    const int64_t n1 = a.all_archive ? a.A : a.nrows;
    const int64_t Nall = n1 + (a.add_recent ? a.T - a.A : 0);
    const int64_t per = (Nall + a.nsplit - 1) / a.nsplit;
    const int64_t pbeg = min(Nall, (int64_t)sp * per);
    const int64_t N = min(Nall, pbeg + per);   // this block's list positions: [pbeg, N)
    const uint16_t* cb = a.cache + (int64_t)b * a.cbs;
    auto row_of = [&](int64_t p) -> int64_t {
        return p < n1 ? (a.all_archive ? p : (int64_t)a.rows[(int64_t)b * a.nrows + p]) : a.A + (p - n1);
    };
    if (lane < 16) {
        s_cnt[lane] = 0;
        s_over[lane] = 0;
    }
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
    float qub[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) qub[i] = sqrtf(__shfl(qs, 4 * g + i) * (1.0f + 0x1p-12f)) * (1.0f + 0x1p-20f);
    constexpr float KE = 2.0f * (float)(D_ROW + D_ROW / 32) * 0x1p-23f;
    float M[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    __builtin_amdgcn_wave_barrier();

    // this lane's row of the tile at list position p0 (clamped to the range),
    // as a 32-bit value that is widened only where it is used, so that the
    // index load can stay in flight
    auto row_at = [&](int64_t p0) -> int32_t {
        const int64_t p = min(p0 + c, N - 1);
        int32_t v = (int32_t)(p < n1 ? p : a.A + (p - n1));
        if (!a.all_archive && p < n1) v = a.rows[(int64_t)b * a.nrows + p];
        return v;
    };
    auto load_rows = [&](int32_t u, bf16x8_t (&xf)[RM_KS]) {
        const uint16_t* src = cb + (int64_t)u * a.cs + 8 * g;
#pragma unroll
        for (int ks = 0; ks < RM_KS; ++ks) xf[ks] = *reinterpret_cast<const bf16x8_t*>(src + 32 * ks);
    };
    // One tile (rows uc, data xc).  The wait at its start drains every load
    // in flight: the tile's own rows and the row indices of the next tile,
    // both issued a tile earlier.  Then the row indices two tiles ahead (unn)
    // and the next tile's rows (xn, rows un) go out and are in flight while
    // this one is scored.  The two row buffers swap roles from tile to tile,
    // so no register copy waits for a load, and the explicit wait tells the
    // compiler that nothing older is outstanding.
    auto score_tile = [&](int64_t p0, bf16x8_t (&xc)[RM_KS], int32_t uc, bf16x8_t (&xn)[RM_KS], int32_t un,
                          int32_t& unn) {
        __builtin_amdgcn_s_waitcnt(VMCNT0);
        unn = p0 + 32 < N ? row_at(p0 + 32) : 0;
        if (p0 + 16 < N) load_rows(un, xn);
        const bool valid = p0 + c < N;
        f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
        float xs = 0.f;
#pragma unroll
        for (int ks = 0; ks < RM_KS; ++ks) {
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[ks], xc[ks], acc, 0, 0, 0);
            xs += sumsq8(xc[ks]);
        }
        xs += __shfl_xor(xs, 16);
        xs += __shfl_xor(xs, 32);
        const float xub = sqrtf(xs * (1.0f + 0x1p-12f)) * (1.0f + 0x1p-20f);
        float lo[4], hi[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float e = next_up_f32(KE * qub[i] * xub * (1.0f + 0x1p-20f) + (float)D_ROW * 0x1p-120f);
            lo[i] = valid ? next_down_f32(acc[i] - e) : -INFINITY;
            hi[i] = valid ? next_up_f32(acc[i] + e) : -INFINITY;
            // running certified lower bound of the maximum: over the 16 rows of the tile (lanes of the group)
            float m = lo[i];
            m = fmaxf(m, __shfl_xor(m, 1));
            m = fmaxf(m, __shfl_xor(m, 2));
            m = fmaxf(m, __shfl_xor(m, 4));
            m = fmaxf(m, __shfl_xor(m, 8));
            M[i] = fmaxf(M[i], m);
        }
        // rows whose upper bound reaches the running bound join the head's list
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int hl = 4 * g + i;
            const bool cand = hi[i] >= M[i] && valid;
            const uint64_t bal = __ballot(cand);
            const uint32_t gm = (uint32_t)(bal >> (16 * g)) & 0xFFFFu;
            int cnt = s_cnt[hl];
            if (cnt + __popc(gm) > RM_CAND) {
                // prune the entries the running bound has passed (16 lanes, 4 entries each)
                int keep[4];
                int32_t kr[4];
                float ku[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int q = c + 16 * j;
                    kr[j] = s_row[hl][q];
                    ku[j] = s_ub[hl][q];
                    keep[j] = (q < cnt && ku[j] >= M[i]) ? 1 : 0;
                }
                __builtin_amdgcn_wave_barrier();
                int base = 0;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t km = (uint32_t)(__ballot(keep[j]) >> (16 * g)) & 0xFFFFu;
                    if (keep[j]) {
                        const int q = base + __popc(km & ((1u << c) - 1u));
                        s_row[hl][q] = kr[j];
                        s_ub[hl][q] = ku[j];
                    }
                    base += __popc(km);
                }
                cnt = base;
                if (c == 0) s_cnt[hl] = cnt;
                __builtin_amdgcn_wave_barrier();
            }
            if (cand) {
                const int q = cnt + __popc(gm & ((1u << c) - 1u));
                if (q < RM_CAND) {
                    s_row[hl][q] = (int32_t)uc;
                    s_ub[hl][q] = hi[i];
                } else {
                    s_over[hl] = 1;   // more near-ties than the list holds: all rows are evaluated
                }
            }
            if (c == 0) s_cnt[hl] = min(cnt + __popc(gm), RM_CAND);
            __builtin_amdgcn_wave_barrier();
        }
    };
    bf16x8_t xa[RM_KS], xb[RM_KS];
    int32_t ua = 0, ub = 0;
    if (N > pbeg) {
        ua = row_at(pbeg);
        load_rows(ua, xa);
        ub = pbeg + 16 < N ? row_at(pbeg + 16) : 0;
    }
    for (int64_t p0 = pbeg; p0 < N; p0 += 32) {
        int32_t ua2 = 0, ub2 = 0;
        score_tile(p0, xa, ua, xb, ub, ua2);
        if (p0 + 16 >= N) break;
        score_tile(p0 + 16, xb, ub, xa, ua2, ub2);
        ua = ua2;
        ub = ub2;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
    // exact fp64 scores of the candidates that reach the final bound (M is
    // read with constant indices: a dynamic index would move it to scratch
    // memory, whose accesses in the tile loop wait for the prefetched tile)
#pragma unroll 1
    for (int i = 0; i < 4; ++i) {
        const float Mi = i == 0 ? M[0] : (i == 1 ? M[1] : (i == 2 ? M[2] : M[3]));
        const int hl = 4 * g + i, h = h0 + hl;
        const bool hv = h < a.H;
        const int64_t hb = (int64_t)b * a.H + (hv ? h : 0);
        const uint16_t* ql = a.q_lat + hb * D_LAT;
        const uint16_t* qr = a.q_rope + hb * D_ROPE;
        double best = -INFINITY;
        int64_t arg = -1;
        if (hv && N > pbeg) {
            if (!s_over[hl]) {
                const int cnt = s_cnt[hl];
                for (int q = c; q < cnt; q += 16) {
                    if (!(s_ub[hl][q] >= Mi)) continue;
                    const int64_t u = s_row[hl][q];
                    const double v = full_score64(ql, qr, cb + u * a.cs);
                    if (ahead(v, u, best, arg)) {
                        best = v;
                        arg = u;
                    }
                }
            } else {
                for (int64_t p = pbeg + c; p < N; p += 16) {
                    const int64_t u = row_of(p);
                    const double v = full_score64(ql, qr, cb + u * a.cs);
                    if (ahead(v, u, best, arg)) {
                        best = v;
                        arg = u;
                    }
                }
            }
        }
        // (max, lowest row) over the 16 lanes of the group
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
            const double ob = __shfl_xor(best, o);
            const int64_t oa = (int64_t)__shfl_xor((long long)arg, o);
            if (ahead(ob, oa, best, arg) && oa >= 0) {
                best = ob;
                arg = oa;
            }
        }
        if (c == 0 && hv) {
            if (a.nsplit > 1) {
                a.part_v[hb * a.nsplit + sp] = best;
                a.part_u[hb * a.nsplit + sp] = (int32_t)arg;
            } else {
                a.smax[hb] = best;
                a.argmax[hb] = (int32_t)arg;
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
    const unsigned nblk = (unsigned)(((a.H + 15) / 16) * a.B * a.nsplit);
    hipLaunchKernelGGL(row_max_kernel, dim3(nblk), dim3(64), 0, s, a);
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
