// Host-side interface between the C ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "acp.h"

namespace acp {

// Per-block statistics of the gate producer (one entry per 64 gates of a head)
// that stage 1's checks need in place of its own pass over log f.
struct GateStats {
    double abs_sum;           // sum of |log f| as a double-double pair (abs_sum, abs_lo)
    double abs_lo;
    int min_lsb;              // smallest float32 ulp exponent of a nonzero gate
    int flags;                // bit 1: a non-finite gate; bit 5: the chained scan timed out
};

struct PlanArgs {
    const void* Q;
    const void* K;
    const float* log_f;
    bool bf16;
    int B, H, L, d;
    int nchunk;               // norm partials per (head, tensor)
    double log_l_over_eps;    // log L - log eps, +inf for eps = 0
    const float* gamma_q;     // [H] QK-norm scale bounds, or null: U from the row norms
    const float* gamma_k;     // [H]
    bool norms_ready;         // part already holds the chunk maxima (the projection's epilogue)
    const GateStats* gate;    // non-null: c is already in place (the gate producer's
                              // epilogue) and these are its per-head statistics
    double* part;             // [B*H, 2, nchunk]
    float* c;                 // [B*H, L]
    double* u;                // [B*H]
    double* delta;            // [B*H]
    int* row_start;           // [B*H, M]
    int* col_end;             // [B*H, M]
    long long* kept;          // [B*H]
    int* flags;               // [B*H]
};

struct GateArgs {
    const void* X;            // [B*L, Dm] bf16 layer inputs
    const void* W;            // [Dm, H] bf16 gate weights
    const float* bias;        // [H]
    int B, L, Dm, H;
    float* log_f;             // [B*H, L]
    float* c;                 // [B*H, L]
    unsigned long long* agg;  // [B*H, L/64, 2] block totals (float64 bits of hi, lo)
    unsigned long long* incl; // [B*H, L/64, 2] inclusive prefixes (float64 bits of hi, lo)
    GateStats* stats;         // [B*H, L/64]
    void* wq;                 // [ceil(H/4), Dm] float4: the weights by group of 4 heads
};

struct FwdArgs {
    const void* Q;
    const void* K;
    const void* V;
    bool bf16;
    int B, H, L, d;
    const float* c;
    const int* row_start;
    const double* u;          // [B*H] logit bound U
    const int* sched;         // [B*H*nb] query-block schedule (bh * nb + block)
    void* O;
    float* lse;
    float* lse2;
};

struct BwdArgs {
    const void* Q;
    const void* K;
    const void* V;
    const void* O;            // the forward's output
    const void* dO;
    bool bf16;
    int B, H, L, d;
    const float* c;
    const int* row_start;
    const int* col_end;
    const float* lse2;
    const int* sched_q;       // query-block schedule (dQ pass)
    const int* sched_k;       // key-block schedule (dK/dV pass)
    float* dsum;              // Delta (float32 path), then Delta' from the dQ pass
    float* rowsum;
    float* colsum;
    void* dQ;
    void* dK;
    void* dV;
    float* dlog_f;
};

struct ProjectArgs {
    const void* X;            // [B*L, Dm] bf16
    const void* Wq;           // [Dm, H*d] bf16
    const void* Wk;
    int B, L, Dm, H, d;
    void* Q;                  // [B, H, L, d] bf16
    void* K;
    double* part;             // [B*H, 2, nchunk] chunk maxima of the squared row norms
    int nchunk;
};

struct DecodeInitArgs {
    const void* K;            // [B*H, L0, d] prompt keys
    const void* V;
    const float* log_f;       // [B*H, L0]
    const float* gamma_q;     // [H]
    const float* gamma_k;     // [H]
    bool bf16;
    int B, H, L0, C, d;
    double log_lmax_over_eps; // log L_max - log eps, +inf for eps = 0
    void* Kc;                 // [B*H, C, d] ring caches, position j in slot j mod C
    void* Vc;
    float* cc;                // [B*H, C] c of the cached positions
    double* cs;               // [2][B*H][2] running sum of log f, (hi, lo) (copy p mod 2
                              // holds the value after position p)
    int* ptr;                 // [2][B*H] first kept block of query p, likewise
    double* delta;            // [B*H]
    int* flags;               // [B*H]
};

struct DecodeArgs {
    const void* q;            // [B*H, d] the new token
    const void* k;
    const void* v;
    const float* log_f;       // [B*H]
    bool bf16;
    int B, H, t, C, d;        // t: position of the new token
    void* Kc;
    void* Vc;
    float* cc;
    double* cs;
    int* ptr;
    const double* delta;
    int* flags;
    float* part;              // split partials: [B*H, nsplit, 2] (max, sum), then
                              // [B*H, nsplit, d] (unnormalised O)
    void* O;                  // [B*H, d]
    float* lse;               // [B*H]
};

// Records the message that acp_last_error() returns and passes the status on.
acp_status set_error(acp_status s, const char* fmt, ...);

// Tracing hooks: no-ops unless acp_timing_enable(1) was called.
void trace_begin(int kernel, hipStream_t s);
void trace_end(int kernel, hipStream_t s);

int norm_chunks(int L);
// Which (head, 128-row block) each logical workgroup id of the attention kernels
// takes: per XCD, heads placed by kept count when there are few, blocks largest
// first.  Tables of B*H*nb entries bh * nb + block, nb = ceil(L / 128).
hipError_t launch_schedule(const long long* kept, const int* row_start, const int* col_end,
                           int BH, int M, int nb, int* sched_q, int* sched_k, hipStream_t s);
hipError_t launch_plan(const PlanArgs& a, hipStream_t s);
hipError_t launch_gate(const GateArgs& a, hipStream_t s);
hipError_t launch_fwd(const FwdArgs& a, hipStream_t s);
hipError_t launch_bwd(const BwdArgs& a, hipStream_t s);
hipError_t launch_dq_bf16(const BwdArgs& a, hipStream_t s);
hipError_t launch_dkdv_bf16(const BwdArgs& a, hipStream_t s);
hipError_t launch_qk_project(const ProjectArgs& a, hipStream_t s);
size_t decode_partials_floats(int BH, int C, int d);
hipError_t launch_decode_init(const DecodeInitArgs& a, hipStream_t s);
hipError_t launch_decode(const DecodeArgs& a, hipStream_t s);

}  // namespace acp
