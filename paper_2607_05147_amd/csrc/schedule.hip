// Hardware-aware prefix scheduler (Algorithm 1 of the section on
// confidence-scheduled verification) as two gfx950 kernels, so the
// verification step needs no host round trip.
//
// sched_rank (one workgroup per 16 candidates, the whole GPU):
//   1. survival a[r][j] = prod_{i<=j} c[r][i] in fp64, multiplied in
//      increasing j (the same sequence of roundings on every implementation),
//      recomputed by every workgroup into LDS;
//   2. the admission order is descending a, ties by the flat index r*K + j.
//      Instead of sorting, every candidate (a > 0) counts the candidates that
//      come before it in that order -- its position n -- and sums their a in
//      the same pass, which gives tau_n = R + sum_{m<=n} a_(m) directly.
//      Sixteen lanes share a candidate, each taking every 16th key, so a
//      wave's LDS reads are sixteen consecutive doubles (no bank conflicts)
//      broadcast to the four candidates of the wave;
//   3. tau and the flat index are written at position n; workgroup 0 writes
//      the candidate count.
// sched_select (one workgroup):
//   4. Theta_n = tau_n * SPS(R + n + 1); mode 0 stops at the first n whose
//      Theta does not exceed its predecessor's (Theta_{-1} = R * SPS(R)),
//      mode 1 takes the first maximum; mode 2 (the asynchronous scheduler's
//      top-K admission) admits a capacity read from device memory, decided on
//      an earlier step's confidences, and evaluates no throughput at all;
//      the capacity call is mode 1 writing its admitted count;
//   5. len[r] = the largest admitted position of r (admission follows each
//      request's prefix order, since a is non-increasing in j), then cu_q and
//      the token -> request marker.
#include "device_common.h"
#include "kernels.h"

#pragma clang fp contract(off)

namespace dspark {

constexpr int kRankThreads = 256;
constexpr int kRankSlices = 16;  // lanes per candidate
constexpr int kRankCand = kRankThreads / kRankSlices;
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / DSPARK_WAVE;

// workspace: [candidate count | pad to 16 B][tau fp64 x N][flat index int32 x N]
__host__ __device__ constexpr size_t ws_tau_off() { return 16; }
__host__ __device__ constexpr size_t ws_idx_off(int N) { return 16 + (size_t)N * 8; }

size_t schedule_workspace(int R, int K) {
    const size_t N = (size_t)R * (K > 0 ? K : 0);
    const size_t b = 16 + N * 12;
    return (b + 255) & ~(size_t)255;
}

__device__ __forceinline__ double sched_conf(float c) {
    if (!(c > 0.0f)) return 0.0;
    if (c > 1.0f) return 1.0;
    return (double)c;
}

__global__ __launch_bounds__(kRankThreads) void sched_rank(const float* __restrict__ conf, int R,
                                                           int K, unsigned char* __restrict__ ws) {
    extern __shared__ __align__(16) double a_l[];  // [N] survival, then [N] staged confidences
    float* conf_l = reinterpret_cast<float*>(a_l + (R * K > 0 ? R * K : 1));
    __shared__ int s_ncand;
    const int tid = threadIdx.x;
    const int N = R * K;
    if (tid == 0) s_ncand = 0;

    // the confidences, staged with coalesced loads: every load of a chunk is
    // issued before the first is used (indices clamped instead of guarded, so
    // no load waits behind a branch)
    for (int base = 0; base < N; base += kRankThreads * 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = conf[min(base + u * kRankThreads + tid, N - 1)];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = base + u * kRankThreads + tid;
            if (i < N) conf_l[i] = v[u];
        }
    }
    __syncthreads();

    // 1. survival products, one request per thread
    int my_cand = 0;
    for (int r = tid; r < R; r += kRankThreads) {
        double p = 1.0;
#pragma unroll 4
        for (int j = 0; j < K; ++j) {
            p = p * sched_conf(conf_l[r * K + j]);
            a_l[r * K + j] = p;
            my_cand += p > 0.0;
        }
    }
    if (blockIdx.x == 0 && my_cand) atomicAdd(&s_ncand, my_cand);
    __syncthreads();

    // 2. position of each candidate in the admission order, and the sum of
    // the a admitted before it
    const int s = tid % kRankSlices;
    const int x = blockIdx.x * kRankCand + tid / kRankSlices;
    const double ax = x < N ? a_l[x] : 0.0;
    // y comes before x iff a_y > a_x, or a_y == a_x and y < x: over y < x
    // the test is a_y >= a_x, over y > x it is a_y > a_x
    int cnt = 0;
    double sum = 0.0;
    if (ax > 0.0) {
#pragma unroll 8
        for (int i = s; i < x; i += kRankSlices) {
            const double ay = a_l[i];
            const bool b = ay >= ax;
            cnt += b;
            sum = sum + (b ? ay : 0.0);
        }
        const int i1 = x + 1 + ((s - (x + 1)) & (kRankSlices - 1));  // first i > x with i % 16 == s
#pragma unroll 8
        for (int i = i1; i < N; i += kRankSlices) {
            const double ay = a_l[i];
            const bool b = ay > ax;
            cnt += b;
            sum = sum + (b ? ay : 0.0);
        }
    }
#pragma unroll
    for (int o = kRankSlices / 2; o > 0; o >>= 1) {
        cnt += __shfl_xor(cnt, o, DSPARK_WAVE);
        sum = sum + __shfl_xor(sum, o, DSPARK_WAVE);
    }

    // 3. scatter by position
    double* tau = reinterpret_cast<double*>(ws + ws_tau_off());
    int32_t* idx = reinterpret_cast<int32_t*>(ws + ws_idx_off(N));
    if (s == 0 && ax > 0.0) {
        tau[cnt] = (double)R + (sum + ax);
        idx[cnt] = x;
    }
    if (blockIdx.x == 0 && tid == 0) *reinterpret_cast<int32_t*>(ws) = s_ncand;
}

template <int E>
__global__ __launch_bounds__(kSelThreads) void sched_select(
    const unsigned char* __restrict__ ws, int R, int K, const double* __restrict__ sps, int mode,
    const int32_t* __restrict__ cap_in, int32_t* __restrict__ cap_out,
    int32_t* __restrict__ len_out, int32_t* __restrict__ cu_q, int32_t* __restrict__ tok_req) {
    extern __shared__ int32_t lenl[];  // [R]
    __shared__ int s_first;
    __shared__ double s_best_v[kSelWaves];
    __shared__ int s_best_n[kSelWaves];
    __shared__ int s_wave_int[kSelWaves];

    const int tid = threadIdx.x;
    const int lane = tid & (DSPARK_WAVE - 1);
    const int wave = tid / DSPARK_WAVE;
    const int N = R * K;
    const double* tau_s = reinterpret_cast<const double*>(ws + ws_tau_off());
    const int32_t* idx_s = reinterpret_cast<const int32_t*>(ws + ws_idx_off(N));

    // every load up front (positions past the candidate count are read but
    // never used): this thread's positions i0 .. i0 + E - 1, tau at i0 - 1,
    // and SPS(R + n + 1) at each position n, SPS(R + i0) before them
    // (indices are clamped, not guarded, so that no load waits behind a
    // branch; the workspace holds at least 256 bytes and sps at least R + N + 1
    // entries, so every clamped index is in bounds, N = 0 included).  Mode 2
    // has no table (sps may be null) and reads only the flat indices.
    const int i0 = tid * E;
    const int nmax = N > 0 ? N - 1 : 0;
    double tv[E], sv[E];
    int iv[E];
    double tprev = 0.0, sprev = 0.0, theta0 = 0.0;
    if (mode != 2) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            tv[e] = tau_s[min(i0 + e, nmax)];
            sv[e] = sps[min(R + i0 + e + 1, R + N)];
        }
        tprev = tau_s[min(max(i0 - 1, 0), nmax)];
        sprev = sps[min(R + i0, R + N)];
        theta0 = (double)R * sps[R];
    }
#pragma unroll
    for (int e = 0; e < E; ++e) iv[e] = idx_s[min(i0 + e, nmax)];
    const int ncand = *reinterpret_cast<const int32_t*>(ws);  // written by sched_rank, N = 0 too

    for (int r = tid; r < R; r += kSelThreads) lenl[r] = 0;
    if (tid == 0) s_first = ncand;
    __syncthreads();

    // 4. throughput along the greedy path and the stop rule
    int n_adm;
    if (mode == 2) {
        // top-K admission: the first min(capacity, candidates) positions; a
        // negative capacity admits none
        n_adm = min(max(*cap_in, 0), ncand);
    } else if (mode == 0) {
        int first = ncand;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int n = i0 + e;
            if (n >= ncand) break;
            const double th = tv[e] * sv[e];
            const double prev = n == 0 ? theta0 : (e == 0 ? tprev * sprev : tv[e - 1] * sv[e - 1]);
            if (!(th > prev)) {
                first = n;
                break;
            }
        }
        if (first < ncand) atomicMin(&s_first, first);
        __syncthreads();
        n_adm = s_first;
    } else {
        double bv = tid == 0 ? theta0 : -1.0 / 0.0;
        int bn = -1;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int n = i0 + e;
            if (n >= ncand) break;
            const double th = tv[e] * sv[e];
            if (th > bv) {
                bv = th;
                bn = n;
            }
        }
        if (tid != 0 && bn == -1) bn = 0x7fffffff;
#pragma unroll
        for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
            const double ov = __shfl_xor(bv, o, DSPARK_WAVE);
            const int on = __shfl_xor(bn, o, DSPARK_WAVE);
            if (ov > bv || (ov == bv && on < bn)) {
                bv = ov;
                bn = on;
            }
        }
        if (lane == 0) {
            s_best_v[wave] = bv;
            s_best_n[wave] = bn;
        }
        __syncthreads();
        if (tid == 0) {
            double v = s_best_v[0];
            int n = s_best_n[0];
            for (int w = 1; w < kSelWaves; ++w)
                if (s_best_v[w] > v || (s_best_v[w] == v && s_best_n[w] < n)) {
                    v = s_best_v[w];
                    n = s_best_n[w];
                }
            s_first = n + 1;
        }
        __syncthreads();
        n_adm = s_first;
    }

    if (cap_out && tid == 0) *cap_out = n_adm;
    if (!len_out) return;  // the capacity call: no lengths

    // 5. lengths: the largest admitted position of each request
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int n = i0 + e;
        if (n < n_adm) atomicMax(&lenl[iv[e] / K], iv[e] % K + 1);
    }
    __syncthreads();

    // cu_q: exclusive scan of 1 + len over requests (contiguous ranges per thread)
    const int per = (R + kSelThreads - 1) / kSelThreads;
    const int r0 = tid * per;
    const int r1 = min(R, r0 + per);
    int tot = 0;
    for (int r = r0; r < r1; ++r) tot += 1 + lenl[r];
    int iinc = tot;
#pragma unroll
    for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
        const int t = __shfl_up(iinc, o, DSPARK_WAVE);
        if (lane >= o) iinc += t;
    }
    if (lane == DSPARK_WAVE - 1) s_wave_int[wave] = iinc;
    __syncthreads();
    int off = 0;
    for (int w = 0; w < wave; ++w) off += s_wave_int[w];
    off += iinc - tot;
    for (int r = r0; r < r1; ++r) {
        const int q = 1 + lenl[r];
        len_out[r] = lenl[r];
        if (cu_q) cu_q[r] = off;
        if (tok_req)
            for (int t = 0; t < q; ++t) tok_req[off + t] = r;
        off += q;
    }
    if (r1 == R && r0 < r1) {
        if (cu_q) cu_q[R] = off;
    }
    if (tok_req) {
        // total = sum(1 + len) from the scan totals, so every thread can clear the tail
        int total = 0;
        for (int w = 0; w < kSelWaves; ++w) total += s_wave_int[w];
        for (int i = total + tid; i < R * (K + 1); i += kSelThreads) tok_req[i] = -1;
    }
}

template <int E>
static hipError_t launch_select(const unsigned char* ws, int R, int K, const double* sps,
                                int mode, const int32_t* cap_in, int32_t* cap_out, int32_t* len,
                                int32_t* cu_q, int32_t* tok_req, hipStream_t s) {
    hipLaunchKernelGGL(sched_select<E>, dim3(1), dim3(kSelThreads), (size_t)R * 4, s, ws, R, K,
                       sps, mode, cap_in, cap_out, len, cu_q, tok_req);
    return hipGetLastError();
}

hipError_t launch_schedule(const float* conf, int R, int K, const double* sps, int mode,
                           const int32_t* cap_in, int32_t* cap_out, int32_t* len, int32_t* cu_q,
                           int32_t* tok_req, void* ws, hipStream_t s) {
    const int N = R * K;
    unsigned char* w = static_cast<unsigned char*>(ws);
    const size_t lds = (size_t)(N > 0 ? N : 1) * 12;
    if (lds >= 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)sched_rank,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    const int grid = N > 0 ? (N + kRankCand - 1) / kRankCand : 1;
    hipLaunchKernelGGL(sched_rank, dim3(grid), dim3(kRankThreads), lds, s, conf, R, K, w);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // positions per thread of the selection (N <= 8192)
    const int per = (N + kSelThreads - 1) / kSelThreads;
    if (per <= 1) return launch_select<1>(w, R, K, sps, mode, cap_in, cap_out, len, cu_q, tok_req, s);
    if (per <= 2) return launch_select<2>(w, R, K, sps, mode, cap_in, cap_out, len, cu_q, tok_req, s);
    if (per <= 4) return launch_select<4>(w, R, K, sps, mode, cap_in, cap_out, len, cu_q, tok_req, s);
    return launch_select<8>(w, R, K, sps, mode, cap_in, cap_out, len, cu_q, tok_req, s);
}

}  // namespace dspark
