// C ABI of the verification step: argument validation (host only, before any
// HIP call), workspace sizing and kernel dispatch.  See include/dspark.h.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <atomic>
#include <string>

#include "dspark.h"

#include "kernels.h"

namespace {

thread_local std::string g_err;

dspark_status fail(dspark_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

dspark_status ok() {
    g_err.clear();
    return DSPARK_OK;
}

dspark_status hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(DSPARK_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

constexpr int kMaxK = 64;
constexpr int kMaxSchedCand = 8192;
constexpr int kMaxR = 8192;
constexpr int kMaxD = 576;
constexpr int kMaxV = 1 << 20;

dspark::AttnArgs make_attn(const void* q, const void* k_cache, const void* v_cache,
                           const int64_t* k_strides, const int64_t* v_strides,
                           const int32_t* block_table, int max_pages, const int32_t* kv_len,
                           const int32_t* cu_q, int R, int max_q, int Hq, int Hkv, int Dqk, int Dv,
                           int page_size, float scale, dspark_dtype dt, void* out, float* lse) {
    dspark::AttnArgs a;
    a.q = q;
    a.k = k_cache;
    a.v = v_cache;
    for (int i = 0; i < 3; ++i) {
        a.ks[i] = k_strides ? k_strides[i] : 0;
        a.vs[i] = v_strides ? v_strides[i] : 0;
    }
    a.block_table = block_table;
    a.max_pages = max_pages;
    a.kv_len = kv_len;
    a.cu_q = cu_q;
    a.R = R;
    a.max_q = max_q;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.Dqk = Dqk;
    a.Dv = Dv;
    a.page = page_size;
    a.scale = scale;
    a.bf16 = dt == DSPARK_BF16;
    a.out = out;
    a.lse = lse;
    return a;
}

dspark_status check_attn_shape(int R, int max_q, int Hq, int Hkv, int Dqk, int Dv, int max_pages,
                               int page_size, dspark_dtype dt) {
    if (dt != DSPARK_F32 && dt != DSPARK_BF16) return fail(DSPARK_EDTYPE, "dtype %d", (int)dt);
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (max_q < 1 || max_q > kMaxK + 1)
        return fail(DSPARK_EINVAL, "max_q=%d outside [1, %d]", max_q, kMaxK + 1);
    if (Hq < 1 || Hkv < 1) return fail(DSPARK_EINVAL, "Hq=%d Hkv=%d", Hq, Hkv);
    if (Hq % Hkv) return fail(DSPARK_ESHAPE, "Hq=%d not a multiple of Hkv=%d", Hq, Hkv);
    if (Dqk < 8 || Dv < 8 || Dqk > kMaxD || Dv > kMaxD || Dqk % 8 || Dv % 8)
        return fail(DSPARK_EUNSUPPORTED, "head dims Dqk=%d Dv=%d (need multiples of 8 up to %d)",
                    Dqk, Dv, kMaxD);
    if (page_size < 16 || page_size % 16)
        return fail(DSPARK_EUNSUPPORTED, "page_size=%d (need a multiple of 16)", page_size);
    if (max_pages < 1) return fail(DSPARK_EINVAL, "max_pages=%d", max_pages);
    if ((int64_t)max_pages * page_size > (int64_t)1 << 30)
        return fail(DSPARK_EUNSUPPORTED, "context bound max_pages*page_size too large");
    const int64_t rows = (int64_t)R * max_q * Hq;
    if (rows * 9 > ((int64_t)1 << 31) - 1)
        return fail(DSPARK_EUNSUPPORTED, "R*max_q*Hq=%lld too large", (long long)rows);
    return DSPARK_OK;
}

}  // namespace

extern "C" {

int dspark_abi_version(void) { return DSPARK_ABI_VERSION; }

const char* dspark_last_error(void) { return g_err.c_str(); }

// ------------------------------------------------------------------ schedule

size_t dspark_schedule_workspace_size(int R, int K) {
    if (R < 1 || R > kMaxR || K < 0 || K > kMaxK || (int64_t)R * K > kMaxSchedCand) return 0;
    return dspark::schedule_workspace(R, K);
}

dspark_status dspark_schedule(const float* conf, int R, int K, const double* sps, int64_t sps_len,
                              int mode, int32_t* len, int32_t* cu_q, int32_t* tok_req, void* ws,
                              size_t ws_bytes, dspark_stream stream) {
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (K < 0 || K > kMaxK) return fail(DSPARK_EINVAL, "K=%d outside [0, %d]", K, kMaxK);
    if ((int64_t)R * K > kMaxSchedCand)
        return fail(DSPARK_EUNSUPPORTED, "R*K=%lld exceeds %d candidates", (long long)R * K,
                    kMaxSchedCand);
    if (mode != 0 && mode != 1) return fail(DSPARK_EINVAL, "mode=%d (0 or 1)", mode);
    if (!len || !sps || (K > 0 && !conf)) return fail(DSPARK_EINVAL, "null conf/sps/len");
    if (sps_len <= (int64_t)R * (K + 1))
        return fail(DSPARK_ESHAPE, "sps_len=%lld must exceed R*(K+1)=%lld", (long long)sps_len,
                    (long long)R * (K + 1));
    if (!aligned(conf, 4) || !aligned(sps, 8) || !aligned(len, 4) || !aligned(cu_q, 4) ||
        !aligned(tok_req, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    const size_t need = dspark::schedule_workspace(R, K);
    if (ws_bytes < need || !ws || !aligned(ws, 256))
        return fail(DSPARK_EWORKSPACE, "workspace of %zu bytes (256-aligned) needed, got %zu",
                    need, ws_bytes);
    return hip_status(dspark::launch_schedule(conf, R, K, sps, mode, nullptr, nullptr, len, cu_q,
                                              tok_req, ws, (hipStream_t)stream),
                      "dspark_schedule");
}

namespace {

dspark_status check_sched_sizes(int R, int K) {
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (K < 0 || K > kMaxK) return fail(DSPARK_EINVAL, "K=%d outside [0, %d]", K, kMaxK);
    if ((int64_t)R * K > kMaxSchedCand)
        return fail(DSPARK_EUNSUPPORTED, "R*K=%lld exceeds %d candidates", (long long)R * K,
                    kMaxSchedCand);
    return DSPARK_OK;
}

dspark_status check_sched_ws(int R, int K, const void* ws, size_t ws_bytes) {
    const size_t need = dspark::schedule_workspace(R, K);
    if (ws_bytes < need || !ws || !aligned(ws, 256))
        return fail(DSPARK_EWORKSPACE, "workspace of %zu bytes (256-aligned) needed, got %zu",
                    need, ws_bytes);
    return DSPARK_OK;
}

}  // namespace

}  // extern "C"

// ------------------------------------------------------------------ no-allocation scheduler

namespace {

// Scratch memory of dspark_schedule_noalloc: the scheduler workspace for the
// largest schedule the ABI accepts (R*K = 8192 candidates), one copy on each
// GPU the library runs on, held until the process ends.
constexpr size_t kNoAllocScratchBytes = ((16 + 12 * (size_t)kMaxSchedCand) + 255) & ~(size_t)255;
constexpr int kMaxDevices = 64;
// Device address of `scratch` on each GPU, looked up once per device.
std::atomic<void*> g_scratch_addr[kMaxDevices];

}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

// Device address of `scratch` on `dev`, looked up with that device current.
// The host-side name `scratch` is not a device address; only this value is
// handed to kernels.
dspark_status scratch_on(int dev, void** out) {
    if (dev < 0 || dev >= kMaxDevices)
        return fail(DSPARK_EUNSUPPORTED, "device %d outside [0, %d)", dev, kMaxDevices);
    void* ptr = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (!ptr) {
        int cur = 0;
        hipError_t e = hipGetDevice(&cur);
        if (e != hipSuccess) return hip_status(e, "hipGetDevice");
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return hip_status(e, "hipSetDevice");
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur != dev) {
            hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess) e = e2;
        }
        if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
        if (!ptr) return fail(DSPARK_EHIP, "hipGetSymbolAddress(scratch) returned null");
        g_scratch_addr[dev].store(ptr, std::memory_order_release);
    }
    *out = ptr;
    return DSPARK_OK;
}

}  // namespace

extern "C" {

dspark_status dspark_schedule_noalloc(const float* conf, int R, int K, const double* sps,
                                      int64_t sps_len, int mode, int32_t* len, int32_t* cu_q,
                                      int32_t* tok_req, dspark_stream stream) {
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (K < 0 || K > kMaxK) return fail(DSPARK_EINVAL, "K=%d outside [0, %d]", K, kMaxK);
    if ((int64_t)R * K > kMaxSchedCand)
        return fail(DSPARK_EUNSUPPORTED, "R*K=%lld exceeds %d candidates", (long long)R * K,
                    kMaxSchedCand);
    if (mode != 0 && mode != 1) return fail(DSPARK_EINVAL, "mode=%d (0 or 1)", mode);
    if (!len || !sps || (K > 0 && !conf)) return fail(DSPARK_EINVAL, "null conf/sps/len");
    if (sps_len <= (int64_t)R * (K + 1))
        return fail(DSPARK_ESHAPE, "sps_len=%lld must exceed R*(K+1)=%lld", (long long)sps_len,
                    (long long)R * (K + 1));
    if (!aligned(conf, 4) || !aligned(sps, 8) || !aligned(len, 4) || !aligned(cu_q, 4) ||
        !aligned(tok_req, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    const size_t need = dspark::schedule_workspace(R, K);
    if (need > kNoAllocScratchBytes)
        return fail(DSPARK_EWORKSPACE, "needs %zu bytes of scratch; the fixed maximum is %zu",
                    need, kNoAllocScratchBytes);
    hipDevice_t dev = 0;
    hipError_t e = hipStreamGetDevice((hipStream_t)stream, &dev);
    if (e != hipSuccess) return hip_status(e, "hipStreamGetDevice");
    void* ws = nullptr;
    if (dspark_status st = scratch_on((int)dev, &ws)) return st;
    // the scheduler writes every workspace value it reads, so nothing is cleared
    return hip_status(dspark::launch_schedule(conf, R, K, sps, mode, nullptr, nullptr, len, cu_q,
                                              tok_req, ws, (hipStream_t)stream),
                      "dspark_schedule_noalloc");
}

dspark_status dspark_schedule_capacity(const float* conf_prev, int R, int K, const double* sps,
                                       int64_t sps_len, int32_t* capacity, void* ws,
                                       size_t ws_bytes, dspark_stream stream) {
    if (dspark_status st = check_sched_sizes(R, K)) return st;
    if (!capacity || !sps || (K > 0 && !conf_prev))
        return fail(DSPARK_EINVAL, "null conf_prev/sps/capacity");
    if (sps_len <= (int64_t)R * (K + 1))
        return fail(DSPARK_ESHAPE, "sps_len=%lld must exceed R*(K+1)=%lld", (long long)sps_len,
                    (long long)R * (K + 1));
    if (!aligned(conf_prev, 4) || !aligned(sps, 8) || !aligned(capacity, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    if (dspark_status st = check_sched_ws(R, K, ws, ws_bytes)) return st;
    return hip_status(dspark::launch_schedule(conf_prev, R, K, sps, 1, nullptr, capacity, nullptr,
                                              nullptr, nullptr, ws, (hipStream_t)stream),
                      "dspark_schedule_capacity");
}

dspark_status dspark_schedule_topk(const float* conf, int R, int K, const int32_t* capacity,
                                   int32_t* len, int32_t* cu_q, int32_t* tok_req, void* ws,
                                   size_t ws_bytes, dspark_stream stream) {
    if (dspark_status st = check_sched_sizes(R, K)) return st;
    if (!capacity || !len || (K > 0 && !conf))
        return fail(DSPARK_EINVAL, "null conf/capacity/len");
    if (!aligned(conf, 4) || !aligned(capacity, 4) || !aligned(len, 4) || !aligned(cu_q, 4) ||
        !aligned(tok_req, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    if (dspark_status st = check_sched_ws(R, K, ws, ws_bytes)) return st;
    return hip_status(dspark::launch_schedule(conf, R, K, nullptr, 2, capacity, nullptr, len,
                                              cu_q, tok_req, ws, (hipStream_t)stream),
                      "dspark_schedule_topk");
}

// ------------------------------------------------------------------ verify attention

size_t dspark_verify_attn_workspace_size(int R, int max_q, int Hq, int Hkv, int Dqk, int Dv,
                                         int max_pages, int page_size, dspark_dtype dt) {
    if (check_attn_shape(R, max_q, Hq, Hkv, Dqk, Dv, max_pages, page_size, dt) != DSPARK_OK)
        return 0;
    // aligned placeholder pointers / dense strides: the size depends on the path only
    const int64_t ks[3] = {(int64_t)Hkv * page_size * Dqk, (int64_t)page_size * Dqk, Dqk};
    const int64_t vs[3] = {(int64_t)Hkv * page_size * Dv, (int64_t)page_size * Dv, Dv};
    const void* fake = (const void*)(uintptr_t)256;
    dspark::AttnArgs a = make_attn(fake, fake, fake, ks, vs, nullptr, max_pages, nullptr, nullptr,
                                   R, max_q, Hq, Hkv, Dqk, Dv, page_size, 1.0f, dt, nullptr,
                                   nullptr);
    size_t need = dspark::attn_generic_workspace(a);
    if (dspark::attn_mfma_supported(a)) need = std::max(need, dspark::attn_mfma_workspace(a));
    if (dspark::attn_mla_shape_ok(a)) need = std::max(need, dspark::attn_mla_workspace(a));
    return need;
}

dspark_status dspark_verify_attn(const void* q, const void* k_cache, const void* v_cache,
                                 const int64_t* k_strides, const int64_t* v_strides,
                                 const int32_t* block_table, int max_pages, const int32_t* kv_len,
                                 const int32_t* cu_q, int R, int max_q, int Hq, int Hkv, int Dqk,
                                 int Dv, int page_size, float scale, dspark_dtype dt, void* out,
                                 float* lse, void* ws, size_t ws_bytes, dspark_stream stream) {
    dspark_status st =
        check_attn_shape(R, max_q, Hq, Hkv, Dqk, Dv, max_pages, page_size, dt);
    if (st != DSPARK_OK) return st;
    if (!q || !k_cache || !v_cache || !k_strides || !v_strides || !block_table || !kv_len ||
        !cu_q || !out)
        return fail(DSPARK_EINVAL, "null argument");
    for (int i = 0; i < 3; ++i)
        if (k_strides[i] < 0 || v_strides[i] < 0)
            return fail(DSPARK_EINVAL, "negative stride");
    if (k_strides[2] < Dqk || v_strides[2] < Dv)
        return fail(DSPARK_ESHAPE, "token stride smaller than the head dim");
    // the kernels take each row's running maximum over raw scores and scale it
    // afterwards, which is the maximum of the scaled scores only for scale > 0
    if (!isfinite(scale) || !(scale > 0.0f))
        return fail(DSPARK_EINVAL, "scale=%g (must be finite and > 0)", (double)scale);
    const size_t esz = dt == DSPARK_BF16 ? 2 : 4;
    if (!aligned(q, esz) || !aligned(k_cache, esz) || !aligned(v_cache, esz) ||
        !aligned(out, esz) || !aligned(lse, 4) || !aligned(block_table, 4) ||
        !aligned(kv_len, 4) || !aligned(cu_q, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    dspark::AttnArgs a = make_attn(q, k_cache, v_cache, k_strides, v_strides, block_table,
                                   max_pages, kv_len, cu_q, R, max_q, Hq, Hkv, Dqk, Dv, page_size,
                                   scale, dt, out, lse);
    // matrix-core paths first: GQA head dim 128, then latent 576/512; else vector ALUs
    const int path = dspark::attn_mfma_supported(a) ? 0 : (dspark::attn_mla_supported(a) ? 1 : 2);
    const size_t need = path == 0 ? dspark::attn_mfma_workspace(a)
                                  : (path == 1 ? dspark::attn_mla_workspace(a)
                                               : dspark::attn_generic_workspace(a));
    if (ws_bytes < need || (need > 0 && !ws) || !aligned(ws, 256))
        return fail(DSPARK_EWORKSPACE, "workspace of %zu bytes (256-aligned) needed, got %zu",
                    need, ws_bytes);
    hipStream_t s = (hipStream_t)stream;
    return hip_status(path == 0 ? dspark::launch_attn_mfma(a, ws, s)
                                : (path == 1 ? dspark::launch_attn_mla(a, ws, s)
                                             : dspark::launch_attn_generic(a, ws, s)),
                      "dspark_verify_attn");
}

// ------------------------------------------------------------------ acceptance

size_t dspark_accept_workspace_size(int R, int K, int V) {
    if (R < 1 || R > kMaxR || K < 0 || K > kMaxK || V < 1 || V > kMaxV) return 0;
    return dspark::accept_workspace(R, K, V);
}

dspark_status dspark_accept(const int32_t* draft_tok, const float* draft_p, const void* logits,
                            dspark_dtype logit_dt, int64_t ld, const float* u,
                            const int32_t* cu_q, int R, int K, int V, float inv_temperature,
                            int32_t* accepted_len, int32_t* next_tok, float* accept_rate,
                            void* ws, size_t ws_bytes, dspark_stream stream) {
    if (logit_dt != DSPARK_F32 && logit_dt != DSPARK_BF16)
        return fail(DSPARK_EDTYPE, "logit dtype %d", (int)logit_dt);
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (K < 0 || K > kMaxK) return fail(DSPARK_EINVAL, "K=%d outside [0, %d]", K, kMaxK);
    if (V < 1 || V > kMaxV) return fail(DSPARK_EINVAL, "V=%d outside [1, %d]", V, kMaxV);
    if (ld < V) return fail(DSPARK_ESHAPE, "ld=%lld smaller than V=%d", (long long)ld, V);
    if (!(inv_temperature > 0.0f) || !isfinite(inv_temperature))
        return fail(DSPARK_EINVAL, "inv_temperature must be positive and finite");
    if (!logits || !cu_q || !accepted_len || !next_tok || (K > 0 && !draft_tok))
        return fail(DSPARK_EINVAL, "null argument");
    // (with K = 0 there is no draft distribution to give: draft_p may be null)
    const bool greedy = draft_p == nullptr && u == nullptr;
    if (!greedy && (u == nullptr || (K > 0 && draft_p == nullptr)))
        return fail(DSPARK_EINVAL, "draft_p and u must both be given (stochastic) or both null");
    if (greedy && accept_rate)
        return fail(DSPARK_EINVAL, "accept_rate needs draft distributions (stochastic mode)");
    const size_t esz = logit_dt == DSPARK_BF16 ? 2 : 4;
    if (!aligned(logits, esz) || !aligned(draft_tok, 4) || !aligned(draft_p, 4) ||
        !aligned(u, 4) || !aligned(cu_q, 4) || !aligned(accepted_len, 4) ||
        !aligned(next_tok, 4) || !aligned(accept_rate, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    const size_t need = dspark::accept_workspace(R, K, V);
    if (ws_bytes < need || !ws || !aligned(ws, 256))
        return fail(DSPARK_EWORKSPACE, "workspace of %zu bytes (256-aligned) needed, got %zu",
                    need, ws_bytes);
    dspark::AcceptArgs a;
    a.draft_tok = draft_tok;
    a.draft_p = draft_p;
    a.logits = logits;
    a.logit_bf16 = logit_dt == DSPARK_BF16;
    a.ld = ld;
    a.u = u;
    a.cu_q = cu_q;
    a.R = R;
    a.K = K;
    a.V = V;
    a.inv_temp = inv_temperature;
    a.accepted_len = accepted_len;
    a.next_tok = next_tok;
    a.accept_rate = accept_rate;
    return hip_status(dspark::launch_accept(a, ws, (hipStream_t)stream), "dspark_accept");
}

size_t dspark_markov_draft_workspace_size(int R, int K, int V, int rank) {
    if (R < 1 || R > kMaxR || K < 1 || K > kMaxK || V < 1 || V > dspark::markov_max_vocab() ||
        !dspark::markov_rank_supported(rank))
        return 0;
    return dspark::markov_workspace(R, K, V, rank);
}

dspark_status dspark_markov_draft(const int32_t* anchor, const void* base_logits,
                                  dspark_dtype base_dt, int64_t ld, const uint16_t* W1,
                                  const uint16_t* W2t, int rank, const uint16_t* hidden,
                                  const float* w_conf, int d, const float* sts_temp,
                                  const float* u, float inv_temperature, int R, int K, int V,
                                  int32_t* draft_tok, float* draft_p, float* conf, void* ws,
                                  size_t ws_bytes, dspark_stream stream) {
    if (base_dt != DSPARK_F32 && base_dt != DSPARK_BF16)
        return fail(DSPARK_EDTYPE, "base logit dtype %d", (int)base_dt);
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (K < 1 || K > kMaxK) return fail(DSPARK_EINVAL, "K=%d outside [1, %d]", K, kMaxK);
    if (V < 1 || V > kMaxV) return fail(DSPARK_EINVAL, "V=%d outside [1, %d]", V, kMaxV);
    if (ld < V) return fail(DSPARK_ESHAPE, "ld=%lld smaller than V=%d", (long long)ld, V);
    if (V > dspark::markov_max_vocab())
        return fail(DSPARK_EUNSUPPORTED, "V=%d above %d", V, dspark::markov_max_vocab());
    if (!dspark::markov_rank_supported(rank))
        return fail(DSPARK_EUNSUPPORTED, "rank=%d (32, 64, 128 or 256)", rank);
    if (d < 0 || d > (1 << 16)) return fail(DSPARK_EINVAL, "d=%d outside [0, 65536]", d);
    if (!(inv_temperature > 0.0f) || !isfinite(inv_temperature))
        return fail(DSPARK_EINVAL, "inv_temperature must be positive and finite");
    if (!anchor || !base_logits || !W1 || !W2t || !w_conf || !u || !draft_tok || !draft_p ||
        !conf || (d > 0 && !hidden))
        return fail(DSPARK_EINVAL, "null argument");
    const size_t esz = base_dt == DSPARK_BF16 ? 2 : 4;
    if (!aligned(W1, 16) || !aligned(W2t, 16))
        return fail(DSPARK_EUNSUPPORTED, "W1 and W2t must be 16-byte aligned");
    if (!aligned(anchor, 4) || !aligned(base_logits, esz) || !aligned(hidden, 2) ||
        !aligned(w_conf, 4) || !aligned(sts_temp, 4) || !aligned(u, 4) ||
        !aligned(draft_tok, 4) || !aligned(draft_p, 4) || !aligned(conf, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    const size_t need = dspark::markov_workspace(R, K, V, rank);
    if (ws_bytes < need || !ws || !aligned(ws, 256))
        return fail(DSPARK_EWORKSPACE, "workspace of %zu bytes (256-aligned) needed, got %zu",
                    need, ws_bytes);
    dspark::MarkovArgs a;
    a.anchor = anchor;
    a.base = base_logits;
    a.base_bf16 = base_dt == DSPARK_BF16;
    a.ld = ld;
    a.W1 = W1;
    a.W2t = W2t;
    a.rank = rank;
    a.hidden = d > 0 ? hidden : nullptr;
    a.w_conf = w_conf;
    a.d = d;
    a.sts_temp = sts_temp;
    a.u = u;
    a.inv_temp = inv_temperature;
    a.R = R;
    a.K = K;
    a.V = V;
    a.draft_tok = draft_tok;
    a.draft_p = draft_p;
    a.conf = conf;
    a.Wrnn = nullptr;
    return hip_status(dspark::launch_markov(a, ws, (hipStream_t)stream), "dspark_markov_draft");
}

size_t dspark_rnn_draft_workspace_size(int R, int K, int V, int rank) {
    if (R < 1 || R > kMaxR || K < 1 || K > kMaxK || V < 1 || V > dspark::markov_max_vocab() ||
        !dspark::markov_rank_supported(rank))
        return 0;
    return dspark::rnn_workspace(R, K, V, rank);
}

dspark_status dspark_rnn_draft(const int32_t* anchor, const void* base_logits,
                               dspark_dtype base_dt, int64_t ld, const uint16_t* W1,
                               const uint16_t* W2t, const uint16_t* Wrnn, int rank,
                               const uint16_t* hidden, const float* w_conf, int d,
                               const float* sts_temp, const float* u, float inv_temperature,
                               int R, int K, int V, int32_t* draft_tok, float* draft_p,
                               float* conf, void* ws, size_t ws_bytes, dspark_stream stream) {
    if (base_dt != DSPARK_F32 && base_dt != DSPARK_BF16)
        return fail(DSPARK_EDTYPE, "base logit dtype %d", (int)base_dt);
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (K < 1 || K > kMaxK) return fail(DSPARK_EINVAL, "K=%d outside [1, %d]", K, kMaxK);
    if (V < 1 || V > kMaxV) return fail(DSPARK_EINVAL, "V=%d outside [1, %d]", V, kMaxV);
    if (ld < V) return fail(DSPARK_ESHAPE, "ld=%lld smaller than V=%d", (long long)ld, V);
    if (V > dspark::markov_max_vocab())
        return fail(DSPARK_EUNSUPPORTED, "V=%d above %d", V, dspark::markov_max_vocab());
    if (!dspark::markov_rank_supported(rank))
        return fail(DSPARK_EUNSUPPORTED, "rank=%d (32, 64, 128 or 256)", rank);
    if (d < 0 || d > (1 << 16)) return fail(DSPARK_EINVAL, "d=%d outside [0, 65536]", d);
    if (d % 8) return fail(DSPARK_EUNSUPPORTED, "d=%d (the RNN head needs a multiple of 8)", d);
    if ((int64_t)R * K > ((int64_t)1 << 24))
        return fail(DSPARK_EUNSUPPORTED, "R*K=%lld too large", (long long)R * K);
    if (!(inv_temperature > 0.0f) || !isfinite(inv_temperature))
        return fail(DSPARK_EINVAL, "inv_temperature must be positive and finite");
    if (!anchor || !base_logits || !W1 || !W2t || !Wrnn || !w_conf || !u || !draft_tok ||
        !draft_p || !conf || (d > 0 && !hidden))
        return fail(DSPARK_EINVAL, "null argument");
    const size_t esz = base_dt == DSPARK_BF16 ? 2 : 4;
    if (!aligned(W1, 16) || !aligned(W2t, 16) || !aligned(Wrnn, 16) ||
        (d > 0 && !aligned(hidden, 16)))
        return fail(DSPARK_EUNSUPPORTED, "W1, W2t, Wrnn and hidden must be 16-byte aligned");
    if (!aligned(anchor, 4) || !aligned(base_logits, esz) || !aligned(w_conf, 4) ||
        !aligned(sts_temp, 4) || !aligned(u, 4) || !aligned(draft_tok, 4) ||
        !aligned(draft_p, 4) || !aligned(conf, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    const size_t need = dspark::rnn_workspace(R, K, V, rank);
    if (ws_bytes < need || !ws || !aligned(ws, 256))
        return fail(DSPARK_EWORKSPACE, "workspace of %zu bytes (256-aligned) needed, got %zu",
                    need, ws_bytes);
    dspark::MarkovArgs a;
    a.anchor = anchor;
    a.base = base_logits;
    a.base_bf16 = base_dt == DSPARK_BF16;
    a.ld = ld;
    a.W1 = W1;
    a.W2t = W2t;
    a.rank = rank;
    a.hidden = d > 0 ? hidden : nullptr;
    a.w_conf = w_conf;
    a.d = d;
    a.sts_temp = sts_temp;
    a.u = u;
    a.inv_temp = inv_temperature;
    a.R = R;
    a.K = K;
    a.V = V;
    a.draft_tok = draft_tok;
    a.draft_p = draft_p;
    a.conf = conf;
    a.Wrnn = Wrnn;
    return hip_status(dspark::launch_rnn(a, ws, (hipStream_t)stream), "dspark_rnn_draft");
}

// ---- input checks ---------------------------------------------------------------

dspark_status dspark_check_verify_inputs(const int32_t* block_table, int max_pages, const int32_t* kv_len,
                                         const int32_t* cu_q, int R, int max_q, int page_size, int num_pages,
                                         int32_t* report, dspark_stream stream) {
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (max_q < 1 || max_pages < 1 || page_size < 1 || num_pages < 1)
        return fail(DSPARK_EINVAL, "max_q=%d max_pages=%d page_size=%d num_pages=%d", max_q, max_pages,
                    page_size, num_pages);
    if ((int64_t)max_pages * page_size > INT32_MAX)
        return fail(DSPARK_EUNSUPPORTED, "context bound max_pages*page_size too large");
    if (!block_table || !kv_len || !cu_q || !report) return fail(DSPARK_EINVAL, "null argument");
    if (!aligned(block_table, 4) || !aligned(kv_len, 4) || !aligned(cu_q, 4) || !aligned(report, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    return hip_status(dspark::launch_check_verify(block_table, max_pages, kv_len, cu_q, R, max_q, page_size,
                                                  num_pages, report, (hipStream_t)stream),
                      "dspark_check_verify_inputs");
}

dspark_status dspark_check_accept_inputs(const int32_t* cu_q, const float* u, int R, int K, int32_t* report,
                                         dspark_stream stream) {
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (K < 0 || K > kMaxK) return fail(DSPARK_EINVAL, "K=%d outside [0, %d]", K, kMaxK);
    if (!cu_q || !report) return fail(DSPARK_EINVAL, "null argument");
    if (!aligned(cu_q, 4) || !aligned(u, 4) || !aligned(report, 4)) return fail(DSPARK_EINVAL, "misaligned pointer");
    return hip_status(dspark::launch_check_accept(cu_q, u, R, K, report, (hipStream_t)stream),
                      "dspark_check_accept_inputs");
}

dspark_status dspark_check_schedule_inputs(const float* conf, int R, int K, int32_t* report,
                                           dspark_stream stream) {
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (K < 0 || K > kMaxK) return fail(DSPARK_EINVAL, "K=%d outside [0, %d]", K, kMaxK);
    if ((K > 0 && !conf) || !report) return fail(DSPARK_EINVAL, "null argument");
    if (!aligned(conf, 4) || !aligned(report, 4)) return fail(DSPARK_EINVAL, "misaligned pointer");
    return hip_status(dspark::launch_check_schedule(conf, R, K, report, (hipStream_t)stream),
                      "dspark_check_schedule_inputs");
}

dspark_status dspark_check_draft_inputs(const float* u, const float* sts_temp, int R, int K, int32_t* report,
                                        dspark_stream stream) {
    if (R < 1 || R > kMaxR) return fail(DSPARK_EINVAL, "R=%d outside [1, %d]", R, kMaxR);
    if (K < 1 || K > kMaxK) return fail(DSPARK_EINVAL, "K=%d outside [1, %d]", K, kMaxK);
    if (!u || !report) return fail(DSPARK_EINVAL, "null argument");
    if (!aligned(u, 4) || !aligned(sts_temp, 4) || !aligned(report, 4))
        return fail(DSPARK_EINVAL, "misaligned pointer");
    return hip_status(dspark::launch_check_draft(u, sts_temp, R, K, report, (hipStream_t)stream),
                      "dspark_check_draft_inputs");
}

}  // extern "C"
