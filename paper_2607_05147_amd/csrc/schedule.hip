// Hardware-aware prefix scheduler (Algorithm 1 of the section on
// confidence-scheduled verification) as one gfx950 workgroup.
//
// Steps, all on the device so the verification step needs no host round trip:
//   1. survival a[r][j] = prod_{i<=j} c[r][i] (fp64, multiplied in increasing j;
//      the same sequence of roundings on every implementation);
//   2. sort of the R*K candidates, descending a, ties by (r, j): the key is the
//      bit pattern of a (non-negative doubles order like their bits) plus the
//      flat index r*K + j.  A merge sort by rank: each request's candidates
//      already form a sorted run, and each level merges runs pairwise with
//      one binary search per candidate (E = Np/1024 candidates per thread);
//   3. block-wide fp64 inclusive scan of the sorted a: tau_n = R + sum_{m<=n} a_m;
//   4. Theta_n = tau_n * SPS(R + n + 1); mode 0 stops at the first n whose Theta
//      does not exceed its predecessor's (Theta_{-1} = R * SPS(R)), mode 1 takes
//      the first maximum;
//   5. len[r] = the largest admitted position of r (admission follows each
//      request's prefix order, since a is non-increasing in j), then cu_q and the
//      token -> request marker.
#include "device_common.h"
#include "kernels.h"

#pragma clang fp contract(off)

namespace dspark {

constexpr int kSchedThreads = 1024;
constexpr int kSchedWaves = kSchedThreads / DSPARK_WAVE;

static int next_pow2(int n) {
    int p = 1;
    while (p < n) p <<= 1;
    return p;
}

size_t schedule_lds_bytes(int R, int K) {
    const int N = R * K;
    const int Np = next_pow2(N > 0 ? N : 1);
    size_t b = (size_t)Np * 8 + (size_t)Np * 2;
    b = (b + 15) & ~(size_t)15;
    b += (size_t)R * 4;
    b = (b + 15) & ~(size_t)15;
    b += (size_t)(N > 0 ? N : 1) * 4;  // staged confidences
    return b;
}

__device__ __forceinline__ double sched_conf(float c) {
    if (!(c > 0.0f)) return 0.0;
    if (c > 1.0f) return 1.0;
    return (double)c;
}

// A sort element: the survival probability's bits (hi, lo) and the flat index.
struct SKey {
    uint32_t hi, lo;
    int idx;
};

// "x comes before y": larger a first, equal a by smaller flat index
__device__ __forceinline__ bool before(const SKey& x, const SKey& y) {
    if (x.hi != y.hi) return x.hi > y.hi;
    if (x.lo != y.lo) return x.lo > y.lo;
    return x.idx < y.idx;
}

template <int E>
__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(
    const float* __restrict__ conf, int R, int K, const double* __restrict__ sps, int mode,
    int Np, int32_t* __restrict__ len_out, int32_t* __restrict__ cu_q,
    int32_t* __restrict__ tok_req) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint64_t* key = reinterpret_cast<uint64_t*>(smem);
    uint16_t* idx = reinterpret_cast<uint16_t*>(key + Np);
    const size_t len_off = (((size_t)Np * 10) + 15) & ~(size_t)15;
    int32_t* lenl = reinterpret_cast<int32_t*>(smem + len_off);
    float* confl = reinterpret_cast<float*>(smem + ((len_off + (size_t)R * 4 + 15) & ~(size_t)15));

    __shared__ double s_wave_tot[kSchedWaves];
    __shared__ int s_first;
    __shared__ int s_ncand;
    __shared__ double s_best_v[kSchedWaves];
    __shared__ int s_best_n[kSchedWaves];
    __shared__ int s_wave_int[kSchedWaves];

    const int tid = threadIdx.x;
    const int lane = tid & (DSPARK_WAVE - 1);
    const int wave = tid / DSPARK_WAVE;
    const int N = R * K;
    const int i0 = tid * E;  // this thread's sorted positions i0 .. i0 + E - 1

    // the throughput table at the positions this thread will examine (sorted
    // position n needs SPS(R + n) and SPS(R + n + 1)), loaded while sorting
    double spsv[E + 1];
#pragma unroll
    for (int e = 0; e <= E; ++e) spsv[e] = (i0 + e <= N) ? sps[R + i0 + e] : 0.0;
    const double sps_r = sps[R];

    if (tid == 0) s_ncand = 0;
    // 1. survival products, one request per thread; the confidences are first
    // staged in LDS with coalesced loads
    for (int i = tid; i < N; i += kSchedThreads) confl[i] = conf[i];
    __syncthreads();
    int my_cand = 0;
    for (int r = tid; r < R; r += kSchedThreads) {
        double p = 1.0;
        for (int j0 = 0; j0 < K; j0 += 16) {
            float c[16];
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) c[jj] = j0 + jj < K ? confl[r * K + j0 + jj] : 1.0f;
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) {
                if (j0 + jj >= K) break;
                p = p * sched_conf(c[jj]);
                key[r * K + j0 + jj] = (uint64_t)__double_as_longlong(p);
                idx[r * K + j0 + jj] = (uint16_t)(r * K + j0 + jj);
                my_cand += p > 0.0;
            }
        }
        lenl[r] = 0;
    }
    for (int i = N + tid; i < Np; i += kSchedThreads) {
        key[i] = 0;
        idx[i] = (uint16_t)i;  // unique, after every real candidate of equal key
    }
    if (my_cand) atomicAdd(&s_ncand, my_cand);
    __syncthreads();

    // 2. merge sort by rank.  Runs of S sorted candidates are merged pairwise:
    // a candidate at in-run index li moves to (run pair start) + li + (the
    // number of the partner run's candidates that come before it), found by a
    // branchless binary search of the partner run.  "before" is a strict total
    // order (the flat index breaks every tie; padding slots carry their own
    // position as index), so the new positions form a permutation.  Each
    // request's K candidates are sorted already (a is non-increasing in j), so
    // for a power-of-two K the merging starts at runs of K.
    SKey v[E];
    int pos[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int i = i0 + e;
        const bool in = i < Np;
        const uint64_t kk = in ? key[i] : 0;
        v[e] = SKey{(uint32_t)(kk >> 32), (uint32_t)kk, in ? (int)idx[i] : 0};
        pos[e] = i;
    }
    // (K = 0 has no candidates; S must start at 1 or more for the loop to end)
    for (int S = K > 0 && (K & (K - 1)) == 0 ? K : 1; S < Np; S <<= 1) {
        int cnt[E];
#pragma unroll
        for (int e = 0; e < E; ++e) cnt[e] = 0;
        for (int b = S; b > 0; b >>= 1) {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                if (pos[e] >= Np || cnt[e] + b > S) continue;
                const int pb = (pos[e] & ~(S - 1)) ^ S;  // the partner run's first position
                const int t = pb + cnt[e] + b - 1;
                const uint64_t kk = key[t];
                const SKey o{(uint32_t)(kk >> 32), (uint32_t)kk, (int)idx[t]};
                if (before(o, v[e])) cnt[e] += b;
            }
        }
        __syncthreads();  // every read of this level is done
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if (pos[e] >= Np) continue;
            pos[e] = (pos[e] & ~(2 * S - 1)) + (pos[e] & (S - 1)) + cnt[e];
            key[pos[e]] = ((uint64_t)v[e].hi << 32) | v[e].lo;
            idx[pos[e]] = (uint16_t)v[e].idx;
        }
        __syncthreads();  // the merged runs are visible
    }
    const int ncand = s_ncand;

    // 3. inclusive scan of the sorted survival probabilities (fp64); thread t
    // owns positions i0 .. i0 + E - 1 (E = 1 covers all when Np <= 1024)
    double loc[E];
    double run = 0.0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int n = i0 + e;
        const double a = (n < ncand) ? __longlong_as_double((long long)key[n]) : 0.0;
        run = run + a;
        loc[e] = run;
    }
    // wave inclusive scan of the per-thread totals
    double incl = run;
#pragma unroll
    for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
        const double t = __shfl_up(incl, o, DSPARK_WAVE);
        if (lane >= o) incl = incl + t;
    }
    if (lane == DSPARK_WAVE - 1) s_wave_tot[wave] = incl;
    __syncthreads();
    double wave_off = 0.0;
    for (int w = 0; w < wave; ++w) wave_off = wave_off + s_wave_tot[w];
    const double excl = wave_off + (incl - run);
    const double Rd = (double)R;
    // tau at this thread's positions, and at the position before them
    double tau[E];
#pragma unroll
    for (int e = 0; e < E; ++e) tau[e] = Rd + (excl + loc[e]);
    // Theta of position n - 1 for the first position of each thread: the
    // previous thread's last tau (theta0 for position 0)
    const double tau_prev_last = __shfl_up(tau[E - 1], 1, DSPARK_WAVE);
    __shared__ double s_wave_last_tau[kSchedWaves];
    if (lane == DSPARK_WAVE - 1) s_wave_last_tau[wave] = tau[E - 1];
    if (tid == 0) s_first = ncand;
    __syncthreads();
    const double theta0 = Rd * sps_r;
    double prev_tau = lane > 0 ? tau_prev_last : (wave > 0 ? s_wave_last_tau[wave - 1] : 0.0);

    // 4. throughput along the greedy path and the stop rule
    int n_adm;
    if (mode == 0) {
        int first = ncand;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int n = i0 + e;
            if (n >= ncand) break;
            const double th = tau[e] * spsv[e + 1];
            const double prev = n == 0 ? theta0 : (e == 0 ? prev_tau : tau[e - 1]) * spsv[e];
            if (!(th > prev)) { first = n; break; }
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
            const double th = tau[e] * spsv[e + 1];
            if (th > bv) { bv = th; bn = n; }
        }
        if (tid != 0 && bn == -1) bn = 0x7fffffff;
#pragma unroll
        for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
            const double ov = __shfl_xor(bv, o, DSPARK_WAVE);
            const int on = __shfl_xor(bn, o, DSPARK_WAVE);
            if (ov > bv || (ov == bv && on < bn)) { bv = ov; bn = on; }
        }
        if (lane == 0) { s_best_v[wave] = bv; s_best_n[wave] = bn; }
        __syncthreads();
        if (tid == 0) {
            double v = s_best_v[0];
            int n = s_best_n[0];
            for (int w = 1; w < kSchedWaves; ++w)
                if (s_best_v[w] > v || (s_best_v[w] == v && s_best_n[w] < n)) {
                    v = s_best_v[w];
                    n = s_best_n[w];
                }
            s_first = n + 1;
        }
        __syncthreads();
        n_adm = s_first;
    }

    // 5. lengths: the largest admitted position of each request
    for (int n = tid; n < n_adm; n += kSchedThreads) {
        const int i = idx[n];
        atomicMax(&lenl[i / K], i % K + 1);
    }
    __syncthreads();

    // cu_q: exclusive scan of 1 + len over requests (contiguous ranges per thread)
    const int per = (R + kSchedThreads - 1) / kSchedThreads;
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
    if (R == 0 && tid == 0 && cu_q) cu_q[0] = 0;
    if (tok_req) {
        // total = sum(1 + len) from the scan totals, so every thread can clear the tail
        int total = 0;
        for (int w = 0; w < kSchedWaves; ++w) total += s_wave_int[w];
        for (int i = total + tid; i < R * (K + 1); i += kSchedThreads) tok_req[i] = -1;
    }
}

template <int E>
static hipError_t launch_e(const float* conf, int R, int K, const double* sps, int mode, int Np,
                           size_t lds, int32_t* len, int32_t* cu_q, int32_t* tok_req,
                           hipStream_t s) {
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)schedule_kernel<E>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(schedule_kernel<E>, dim3(1), dim3(kSchedThreads), lds, s, conf, R, K, sps,
                       mode, Np, len, cu_q, tok_req);
    return hipGetLastError();
}

hipError_t launch_schedule(const float* conf, int R, int K, const double* sps, int mode,
                           int32_t* len, int32_t* cu_q, int32_t* tok_req, hipStream_t s) {
    const int N = R * K;
    const int Np = next_pow2(N > 0 ? N : 1);
    const size_t lds = schedule_lds_bytes(R, K);
    // keys per thread (N <= 8192)
    switch (Np <= kSchedThreads ? 1 : Np / kSchedThreads) {
        case 1: return launch_e<1>(conf, R, K, sps, mode, Np, lds, len, cu_q, tok_req, s);
        case 2: return launch_e<2>(conf, R, K, sps, mode, Np, lds, len, cu_q, tok_req, s);
        case 4: return launch_e<4>(conf, R, K, sps, mode, Np, lds, len, cu_q, tok_req, s);
        default: return launch_e<8>(conf, R, K, sps, mode, Np, lds, len, cu_q, tok_req, s);
    }
}

}  // namespace dspark
