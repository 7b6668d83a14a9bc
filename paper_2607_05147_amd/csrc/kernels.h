// Host-side launchers of the gfx950 kernels (defined in the .hip files).
// Arguments are already validated by the C ABI layer.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dspark {

// ---- scheduler --------------------------------------------------------------
size_t schedule_workspace(int R, int K);
// mode 0: early stop; 1: no break; 2: top-K with the capacity *cap_in (device).
// cap_out (device, nullable) receives the admitted count; len == null skips
// the lengths, cu_q and tok_req.
hipError_t launch_schedule(const float* conf, int R, int K, const double* sps, int mode,
                           const int32_t* cap_in, int32_t* cap_out, int32_t* len, int32_t* cu_q,
                           int32_t* tok_req, void* ws, hipStream_t s);

// ---- verify attention ---------------------------------------------------------
struct AttnArgs {
    const void* q;
    const void* k;
    const void* v;
    int64_t ks[3];
    int64_t vs[3];
    const int32_t* block_table;
    int max_pages;
    const int32_t* kv_len;
    const int32_t* cu_q;
    int R, max_q, Hq, Hkv, Dqk, Dv, page;
    float scale;
    int bf16;  // 0 = fp32, 1 = bf16
    void* out;
    float* lse;
};

// The MFMA path handles bf16, Dqk == Dv == 128, page % 32 == 0.
bool attn_mfma_supported(const AttnArgs& a);
size_t attn_mfma_workspace(const AttnArgs& a);
hipError_t launch_attn_mfma(const AttnArgs& a, void* ws, hipStream_t s);
bool attn_mla_shape_ok(const AttnArgs& a);   // shape only (workspace sizing)
bool attn_mla_supported(const AttnArgs& a);  // shape, value aliasing and alignment
size_t attn_mla_workspace(const AttnArgs& a);
hipError_t launch_attn_mla(const AttnArgs& a, void* ws, hipStream_t s);

size_t attn_generic_workspace(const AttnArgs& a);
hipError_t launch_attn_generic(const AttnArgs& a, void* ws, hipStream_t s);

// ---- acceptance ------------------------------------------------------------------
struct AcceptArgs {
    const int32_t* draft_tok;
    const float* draft_p;
    const void* logits;
    int logit_bf16;
    int64_t ld;
    const float* u;
    const int32_t* cu_q;
    int R, K, V;
    float inv_temp;
    int32_t* accepted_len;
    int32_t* next_tok;
    float* accept_rate;
};

size_t accept_workspace(int R, int K, int V);
hipError_t launch_accept(const AcceptArgs& a, void* ws, hipStream_t s);

// ---- Markov-head draft block ----------------------------------------------------
struct MarkovArgs {
    const int32_t* anchor;
    const void* base;  // base logits, row (r * K + k - 1) at element offset row * ld
    int base_bf16;
    int64_t ld;
    const uint16_t* W1;   // [V, rank] bf16
    const uint16_t* W2t;  // [V, rank] bf16, row v = W2[:, v]
    int rank;
    const uint16_t* hidden;  // [R, K, d] bf16 (null when d == 0)
    const float* w_conf;     // [d + rank]
    int d;
    const float* sts_temp;  // [K] or null
    const float* u;         // [R, K]
    float inv_temp;
    int R, K, V;
    int32_t* draft_tok;  // [R, K]
    float* draft_p;      // [R, K, V]
    float* conf;         // [R, K]
    const uint16_t* Wrnn;  // RNN head only: [3 rank, 2 rank + d] bf16 (gate, candidate, output)
};
size_t markov_workspace(int R, int K, int V, int rank);
size_t rnn_workspace(int R, int K, int V, int rank);
hipError_t launch_rnn(const MarkovArgs& a, void* ws, hipStream_t s);
bool markov_rank_supported(int rank);
int markov_max_vocab();  // per-tile statistics of one request fit one workgroup
hipError_t launch_markov(const MarkovArgs& a, void* ws, hipStream_t s);

// ---- input checks (device-side values) -------------------------------------------
hipError_t launch_check_verify(const int32_t* block_table, int max_pages, const int32_t* kv_len,
                               const int32_t* cu_q, int R, int max_q, int page_size, int num_pages,
                               int32_t* report, hipStream_t s);
hipError_t launch_check_accept(const int32_t* cu_q, const float* u, int R, int K, int32_t* report,
                               hipStream_t s);
hipError_t launch_check_schedule(const float* conf, int R, int K, int32_t* report, hipStream_t s);
hipError_t launch_check_draft(const float* u, const float* sts_temp, int R, int K, int32_t* report,
                              hipStream_t s);

}  // namespace dspark
