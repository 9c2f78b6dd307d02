// C ABI of the library: argument validation, workspace layout and launches.
#include "acp.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "acp_internal.h"

namespace {

thread_local std::string g_last_error;

acp_status fail(acp_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

acp_status ok() {
    g_last_error.clear();
    return ACP_OK;
}

struct Layout {
    size_t c, u, delta, rs, ce, kept, flags, part, lse2, dsum, rowsum, colsum, sched_q, sched_k,
        gate_agg, gate_incl, gate_stats, total;
    int nchunk;
};

Layout layout(int B, int H, int L, int d) {
    Layout y{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off += (bytes + 255) & ~(size_t)255;
        return o;
    };
    const size_t BH = (size_t)B * H, BHL = BH * L, M = (size_t)L / 64;
    y.nchunk = acp::norm_chunks(L);
    y.c = take(BHL * 4);
    y.u = take(BH * 8);
    y.delta = take(BH * 8);
    y.rs = take(BH * M * 4);
    y.ce = take(BH * M * 4);
    y.kept = take(BH * 8);
    y.flags = take(BH * 4);
    y.part = take(BH * 2 * (size_t)y.nchunk * 8);
    y.lse2 = take(BHL * 4);
    y.dsum = take(BHL * 4);
    y.rowsum = take(BHL * 4);
    y.colsum = take(BHL * 4);
    const size_t nb = ((size_t)L + 127) / 128;   // 128-row blocks of the attention kernels
    y.sched_q = take(BH * nb * 4);
    y.sched_k = take(BH * nb * 4);
    y.gate_agg = take(BH * M * 16);     // gate producer's chained scan (acp_gate_project):
    y.gate_incl = take(BH * M * 16);    // a double-double pair per block
    y.gate_stats = take(BH * M * sizeof(acp::GateStats));
    y.total = off;
    return y;
}

struct DecLayout {
    size_t k, v, c, cum, delta, ptr, flags, part, total;
};

acp_status check_shape(int B, int H, int L, int d, acp_dtype dt) {
    if (B <= 0 || H <= 0 || L <= 0 || d <= 0)
        return fail(ACP_EINVAL, "sizes must be positive (B=%d H=%d L=%d d=%d)", B, H, L, d);
    if (dt != ACP_F32 && dt != ACP_BF16) return fail(ACP_EINVAL, "unknown dtype %d", (int)dt);
    if (d != 64 && d != 128) return fail(ACP_EUNSUPPORTED, "head dim %d not in {64, 128}", d);
    if (L % 64 != 0) return fail(ACP_EUNSUPPORTED, "L=%d is not a multiple of 64", L);
    if (L > 64 * 2048) return fail(ACP_EUNSUPPORTED, "L=%d exceeds 131072", L);
    if ((long long)B * H > 65535)
        return fail(ACP_EUNSUPPORTED, "B*H=%lld exceeds 65535", (long long)B * H);
    return ACP_OK;
}

acp_status check_ptr(const void* p, const char* name) {
    if (p == nullptr) return fail(ACP_EINVAL, "%s is NULL", name);
    if (((uintptr_t)p & 15) != 0) return fail(ACP_EINVAL, "%s is not 16-byte aligned", name);
    return ACP_OK;
}

acp_status check_eps(double eps) {
    if (!std::isfinite(eps) || eps < 0.0 || eps >= 1.0)
        return fail(ACP_EINVAL, "eps=%g outside [0, 1)", eps);
    return ACP_OK;
}

acp_status check_ws(void* ws, size_t ws_bytes, const Layout& y) {
    acp_status s = check_ptr(ws, "ws");
    if (s != ACP_OK) return s;
    if (ws_bytes < y.total)
        return fail(ACP_EWORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, y.total);
    return ACP_OK;
}

acp_status hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(ACP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define ACP_TRY(expr)                      \
    do {                                   \
        const acp_status s_ = (expr);      \
        if (s_ != ACP_OK) return s_;       \
    } while (0)

double log_l_over_eps(int L, double eps) {
    return eps == 0.0 ? INFINITY : std::log((double)L) - std::log(eps);
}

acp::PlanArgs plan_args(const void* Q, const void* K, const float* log_f, acp_dtype dt, int B,
                        int H, int L, int d, double eps, const Layout& y, char* w) {
    acp::PlanArgs a{};
    a.Q = Q; a.K = K; a.log_f = log_f; a.bf16 = dt == ACP_BF16;
    a.B = B; a.H = H; a.L = L; a.d = d;
    a.nchunk = y.nchunk;
    a.log_l_over_eps = log_l_over_eps(L, eps);
    a.part = (double*)(w + y.part);
    a.c = (float*)(w + y.c);
    a.u = (double*)(w + y.u);
    a.delta = (double*)(w + y.delta);
    a.row_start = (int*)(w + y.rs);
    a.col_end = (int*)(w + y.ce);
    a.kept = (long long*)(w + y.kept);
    a.flags = (int*)(w + y.flags);
    return a;
}

// ---- tracing -------------------------------------------------------------------
struct TraceRec {
    int kernel;
    hipEvent_t start, stop;
};
struct TraceState {
    bool on = false;
    std::vector<hipEvent_t> pool;    // created events, reused after a reset
    size_t next = 0;                 // first unused event in pool
    std::vector<TraceRec> recs;
    int open_kernel = -1;
    hipEvent_t open_start = nullptr;
};
TraceState g_trace;

hipEvent_t trace_event() {
    if (g_trace.next == g_trace.pool.size()) {
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        g_trace.pool.push_back(e);
    }
    return g_trace.pool[g_trace.next++];
}

}  // namespace

namespace acp {
acp_status set_error(acp_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

void trace_begin(int kernel, hipStream_t s) {
    if (!g_trace.on) return;
    hipEvent_t e = trace_event();
    if (e == nullptr) return;
    (void)hipEventRecord(e, s);
    g_trace.open_kernel = kernel;
    g_trace.open_start = e;
}
void trace_end(int kernel, hipStream_t s) {
    if (!g_trace.on || g_trace.open_start == nullptr || g_trace.open_kernel != kernel) return;
    hipEvent_t e = trace_event();
    if (e == nullptr) return;
    (void)hipEventRecord(e, s);
    g_trace.recs.push_back({kernel, g_trace.open_start, e});
    g_trace.open_start = nullptr;
    g_trace.open_kernel = -1;
}
}  // namespace acp

extern "C" {

acp_status acp_timing_enable(int on) {
    g_trace.on = on != 0;
    return ok();
}

acp_status acp_timing_reset(void) {
    g_trace.recs.clear();
    g_trace.next = 0;
    g_trace.open_start = nullptr;
    g_trace.open_kernel = -1;
    return ok();
}

acp_status acp_timing_read(acp_kernel_times* out) {
    if (out == nullptr) return fail(ACP_EINVAL, "out is NULL");
    for (int k = 0; k < ACP_K_COUNT; ++k) {
        out->launches[k] = 0;
        out->ms[k] = 0.0;
    }
    for (const TraceRec& r : g_trace.recs) {
        hipError_t e = hipEventSynchronize(r.stop);
        if (e != hipSuccess) return hip_status(e, "acp_timing_read");
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, r.start, r.stop);
        if (e != hipSuccess) return hip_status(e, "acp_timing_read");
        out->launches[r.kernel] += 1;
        out->ms[r.kernel] += ms;
    }
    return ok();
}

acp_status acp_workspace_size(int B, int H, int L, int d, acp_dtype dt, size_t* bytes) {
    ACP_TRY(check_shape(B, H, L, d, dt));
    if (bytes == nullptr) return fail(ACP_EINVAL, "bytes is NULL");
    *bytes = layout(B, H, L, d).total;
    return ok();
}

acp_status acp_plan_offsets(int B, int H, int L, int d, acp_dtype dt, acp_plan_layout* out) {
    ACP_TRY(check_shape(B, H, L, d, dt));
    if (out == nullptr) return fail(ACP_EINVAL, "out is NULL");
    const Layout y = layout(B, H, L, d);
    out->c = y.c;
    out->bound_u = y.u;
    out->delta = y.delta;
    out->row_start = y.rs;
    out->col_end = y.ce;
    out->kept = y.kept;
    out->flags = y.flags;
    out->sched_q = y.sched_q;
    out->sched_k = y.sched_k;
    out->total = y.total;
    return ok();
}

acp_status acp_boundary(const void* Q, const void* K, const float* log_f, acp_dtype dt, int B,
                        int H, int L, int d, double eps, float* c, double* bound_u,
                        double* delta, int32_t* row_start, int32_t* col_end, int64_t* kept,
                        int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
    ACP_TRY(check_shape(B, H, L, d, dt));
    ACP_TRY(check_eps(eps));
    ACP_TRY(check_ptr(Q, "Q"));
    ACP_TRY(check_ptr(K, "K"));
    ACP_TRY(check_ptr(log_f, "log_f"));
    ACP_TRY(check_ptr(c, "c"));
    ACP_TRY(check_ptr(bound_u, "bound_u"));
    ACP_TRY(check_ptr(delta, "delta"));
    ACP_TRY(check_ptr(row_start, "row_start"));
    ACP_TRY(check_ptr(col_end, "col_end"));
    ACP_TRY(check_ptr(kept, "kept"));
    ACP_TRY(check_ptr(flags, "flags"));
    const Layout y = layout(B, H, L, d);
    ACP_TRY(check_ws(ws, ws_bytes, y));
    acp::PlanArgs a = plan_args(Q, K, log_f, dt, B, H, L, d, eps, y, (char*)ws);
    a.c = c;
    a.u = bound_u;
    a.delta = delta;
    a.row_start = row_start;
    a.col_end = col_end;
    a.kept = (long long*)kept;
    a.flags = flags;
    return hip_status(acp::launch_plan(a, (hipStream_t)stream), "acp_boundary launch");
}

acp_status acp_boundary_qknorm(const float* log_f, const float* gamma_q, const float* gamma_k,
                               acp_dtype dt, int B, int H, int L, int d, double eps, float* c,
                               double* bound_u, double* delta, int32_t* row_start,
                               int32_t* col_end, int64_t* kept, int32_t* flags, void* ws,
                               size_t ws_bytes, void* stream) {
    ACP_TRY(check_shape(B, H, L, d, dt));
    ACP_TRY(check_eps(eps));
    ACP_TRY(check_ptr(log_f, "log_f"));
    ACP_TRY(check_ptr(gamma_q, "gamma_q"));
    ACP_TRY(check_ptr(gamma_k, "gamma_k"));
    ACP_TRY(check_ptr(c, "c"));
    ACP_TRY(check_ptr(bound_u, "bound_u"));
    ACP_TRY(check_ptr(delta, "delta"));
    ACP_TRY(check_ptr(row_start, "row_start"));
    ACP_TRY(check_ptr(col_end, "col_end"));
    ACP_TRY(check_ptr(kept, "kept"));
    ACP_TRY(check_ptr(flags, "flags"));
    const Layout y = layout(B, H, L, d);
    ACP_TRY(check_ws(ws, ws_bytes, y));
    acp::PlanArgs a = plan_args(nullptr, nullptr, log_f, dt, B, H, L, d, eps, y, (char*)ws);
    a.gamma_q = gamma_q;
    a.gamma_k = gamma_k;
    a.c = c;
    a.u = bound_u;
    a.delta = delta;
    a.row_start = row_start;
    a.col_end = col_end;
    a.kept = (long long*)kept;
    a.flags = flags;
    return hip_status(acp::launch_plan(a, (hipStream_t)stream), "acp_boundary_qknorm launch");
}

// Forward after a stage 1 whose bound comes from the row norms (gamma_q null;
// norms_ready: their chunk maxima are already in ws) or from QK-norm scales.
static acp_status fwd_common(const void* Q, const void* K, const void* V, const float* log_f,
                             const float* gamma_q, const float* gamma_k, acp_dtype dt, int B,
                             int H, int L, int d, double eps, void* O, float* lse, void* ws,
                             size_t ws_bytes, void* stream, bool norms_ready = false,
                             bool gated = false) {
    ACP_TRY(check_shape(B, H, L, d, dt));
    ACP_TRY(check_eps(eps));
    ACP_TRY(check_ptr(Q, "Q"));
    ACP_TRY(check_ptr(K, "K"));
    ACP_TRY(check_ptr(V, "V"));
    if (!gated) ACP_TRY(check_ptr(log_f, "log_f"));
    ACP_TRY(check_ptr(O, "O"));
    ACP_TRY(check_ptr(lse, "lse"));
    const Layout y = layout(B, H, L, d);
    ACP_TRY(check_ws(ws, ws_bytes, y));
    char* w = (char*)ws;
    acp::PlanArgs p = plan_args(Q, K, log_f, dt, B, H, L, d, eps, y, w);
    p.gamma_q = gamma_q;
    p.gamma_k = gamma_k;
    p.norms_ready = norms_ready;
    if (gated) p.gate = (const acp::GateStats*)(w + y.gate_stats);
    hipError_t e = acp::launch_plan(p, (hipStream_t)stream);
    if (e != hipSuccess) return hip_status(e, "fox_attn_fwd boundary launch");
    if (dt == ACP_BF16) {
        e = acp::launch_schedule((const long long*)(w + y.kept), (const int*)(w + y.rs),
                                 (const int*)(w + y.ce), B * H, L / 64, (L + 127) / 128,
                                 (int*)(w + y.sched_q), (int*)(w + y.sched_k), (hipStream_t)stream);
        if (e != hipSuccess) return hip_status(e, "fox_attn_fwd schedule launch");
    }
    acp::FwdArgs f{};
    f.Q = Q; f.K = K; f.V = V; f.bf16 = dt == ACP_BF16;
    f.B = B; f.H = H; f.L = L; f.d = d;
    f.c = (const float*)(w + y.c);
    f.row_start = (const int*)(w + y.rs);
    f.u = (const double*)(w + y.u);
    f.sched = (const int*)(w + y.sched_q);
    f.O = O;
    f.lse = lse;
    f.lse2 = (float*)(w + y.lse2);
    return hip_status(acp::launch_fwd(f, (hipStream_t)stream), "fox_attn_fwd launch");
}

acp_status fox_attn_fwd(const void* Q, const void* K, const void* V, const float* log_f,
                        acp_dtype dt, int B, int H, int L, int d, double eps, void* O,
                        float* lse, void* ws, size_t ws_bytes, void* stream) {
    return fwd_common(Q, K, V, log_f, nullptr, nullptr, dt, B, H, L, d, eps, O, lse, ws,
                      ws_bytes, stream);
}

acp_status fox_attn_fwd_qknorm(const void* Q, const void* K, const void* V, const float* log_f,
                               const float* gamma_q, const float* gamma_k, acp_dtype dt, int B,
                               int H, int L, int d, double eps, void* O, float* lse, void* ws,
                               size_t ws_bytes, void* stream) {
    ACP_TRY(check_ptr(gamma_q, "gamma_q"));
    ACP_TRY(check_ptr(gamma_k, "gamma_k"));
    return fwd_common(Q, K, V, log_f, gamma_q, gamma_k, dt, B, H, L, d, eps, O, lse, ws,
                      ws_bytes, stream);
}

acp_status fox_attn_fwd_projected(const void* Q, const void* K, const void* V, const float* log_f,
                                  acp_dtype dt, int B, int H, int L, int d, double eps, void* O,
                                  float* lse, void* ws, size_t ws_bytes, void* stream) {
    return fwd_common(Q, K, V, log_f, nullptr, nullptr, dt, B, H, L, d, eps, O, lse, ws,
                      ws_bytes, stream, true);
}

acp_status acp_gate_project(const void* X, const void* w_f, const float* b_f, int B, int L,
                            int d_model, int H, int d, float* log_f, void* ws, size_t ws_bytes,
                            void* stream) {
    ACP_TRY(check_shape(B, H, L, d, ACP_BF16));
    if (d_model <= 0 || d_model % 64 != 0 || d_model > 8192)
        return fail(ACP_EUNSUPPORTED, "d_model=%d is not a multiple of 64 in [64, 8192]", d_model);
    if (H > 64) return fail(ACP_EUNSUPPORTED, "H=%d: the gate projection takes at most 64 heads", H);
    ACP_TRY(check_ptr(X, "X"));
    ACP_TRY(check_ptr(w_f, "w_f"));
    if (b_f == nullptr) return fail(ACP_EINVAL, "b_f is NULL");
    ACP_TRY(check_ptr(log_f, "log_f"));
    const Layout y = layout(B, H, L, d);
    ACP_TRY(check_ws(ws, ws_bytes, y));
    char* w = (char*)ws;
    acp::GateArgs a{};
    a.X = X; a.W = w_f; a.bias = b_f;
    a.B = B; a.L = L; a.Dm = d_model; a.H = H;
    a.log_f = log_f;
    a.c = (float*)(w + y.c);
    a.agg = (unsigned long long*)(w + y.gate_agg);
    a.incl = (unsigned long long*)(w + y.gate_incl);
    a.stats = (acp::GateStats*)(w + y.gate_stats);
    // the float32 copy of the weights goes where the backward keeps Delta' (free
    // until a backward runs on this workspace)
    const size_t wq_bytes = (size_t)((H + 3) / 4) * d_model * 16;
    if (wq_bytes > (size_t)B * H * L * 4)
        return fail(ACP_EUNSUPPORTED, "d_model=%d too large for these shapes (%zu bytes of "
                    "float32 weights, %zu available)", d_model, wq_bytes, (size_t)B * H * L * 4);
    a.wq = w + y.dsum;
    return hip_status(acp::launch_gate(a, (hipStream_t)stream), "acp_gate_project launch");
}

acp_status fox_attn_fwd_gated(const void* Q, const void* K, const void* V, acp_dtype dt, int B,
                              int H, int L, int d, double eps, void* O, float* lse, void* ws,
                              size_t ws_bytes, void* stream) {
    return fwd_common(Q, K, V, nullptr, nullptr, nullptr, dt, B, H, L, d, eps, O, lse, ws,
                      ws_bytes, stream, false, true);
}

acp_status acp_qk_project(const void* X, const void* Wq, const void* Wk, acp_dtype dt, int B,
                          int L, int d_model, int H, int d, void* Q, void* K, void* ws,
                          size_t ws_bytes, void* stream) {
    ACP_TRY(check_shape(B, H, L, d, dt));
    if (dt != ACP_BF16) return fail(ACP_EUNSUPPORTED, "the projection takes bfloat16 only");
    if (L % 128 != 0) return fail(ACP_EUNSUPPORTED, "L=%d is not a multiple of 128", L);
    if (d_model <= 0 || d_model % 64 != 0)
        return fail(ACP_EUNSUPPORTED, "d_model=%d is not a positive multiple of 64", d_model);
    if ((H * d) % 128 != 0) return fail(ACP_EUNSUPPORTED, "H*d=%d is not a multiple of 128", H * d);
    if ((long long)B * L / 128 > 65535)
        return fail(ACP_EUNSUPPORTED, "B*L=%lld exceeds 8388480", (long long)B * L);
    ACP_TRY(check_ptr(X, "X"));
    ACP_TRY(check_ptr(Wq, "Wq"));
    ACP_TRY(check_ptr(Wk, "Wk"));
    ACP_TRY(check_ptr(Q, "Q"));
    ACP_TRY(check_ptr(K, "K"));
    const Layout y = layout(B, H, L, d);
    ACP_TRY(check_ws(ws, ws_bytes, y));
    acp::ProjectArgs a{};
    a.X = X; a.Wq = Wq; a.Wk = Wk;
    a.B = B; a.L = L; a.Dm = d_model; a.H = H; a.d = d;
    a.Q = Q; a.K = K;
    a.part = (double*)((char*)ws + y.part);
    a.nchunk = y.nchunk;
    return hip_status(acp::launch_qk_project(a, (hipStream_t)stream), "acp_qk_project launch");
}

acp_status fox_attn_bwd(const void* Q, const void* K, const void* V, const void* O,
                        const void* dO, acp_dtype dt, int B, int H, int L, int d, void* dQ,
                        void* dK, void* dV, float* dlog_f, void* ws, size_t ws_bytes,
                        void* stream) {
    ACP_TRY(check_shape(B, H, L, d, dt));
    ACP_TRY(check_ptr(Q, "Q"));
    ACP_TRY(check_ptr(K, "K"));
    ACP_TRY(check_ptr(V, "V"));
    ACP_TRY(check_ptr(O, "O"));
    ACP_TRY(check_ptr(dO, "dO"));
    ACP_TRY(check_ptr(dQ, "dQ"));
    ACP_TRY(check_ptr(dK, "dK"));
    ACP_TRY(check_ptr(dV, "dV"));
    ACP_TRY(check_ptr(dlog_f, "dlog_f"));
    const Layout y = layout(B, H, L, d);
    ACP_TRY(check_ws(ws, ws_bytes, y));
    char* w = (char*)ws;
    acp::BwdArgs b{};
    b.Q = Q; b.K = K; b.V = V; b.O = O; b.dO = dO; b.bf16 = dt == ACP_BF16;
    b.B = B; b.H = H; b.L = L; b.d = d;
    b.c = (const float*)(w + y.c);
    b.row_start = (const int*)(w + y.rs);
    b.col_end = (const int*)(w + y.ce);
    b.lse2 = (const float*)(w + y.lse2);
    b.sched_q = (const int*)(w + y.sched_q);
    b.sched_k = (const int*)(w + y.sched_k);
    b.dsum = (float*)(w + y.dsum);
    b.rowsum = (float*)(w + y.rowsum);
    b.colsum = (float*)(w + y.colsum);
    b.dQ = dQ; b.dK = dK; b.dV = dV; b.dlog_f = dlog_f;
    return hip_status(acp::launch_bwd(b, (hipStream_t)stream), "fox_attn_bwd launch");
}

// ---- decoding ----------------------------------------------------------------------
static DecLayout dec_layout(int B, int H, int C, int d, acp_dtype dt) {
    DecLayout y{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off += (bytes + 255) & ~(size_t)255;
        return o;
    };
    const size_t BH = (size_t)B * H, es = dt == ACP_BF16 ? 2 : 4;
    y.k = take(BH * C * d * es);
    y.v = take(BH * C * d * es);
    y.c = take(BH * C * 4);
    y.cum = take(2 * BH * 16);
    y.delta = take(BH * 8);
    y.ptr = take(2 * BH * 4);
    y.flags = take(BH * 4);
    y.part = take(acp::decode_partials_floats((int)BH, C, d) * 4);
    y.total = off;
    return y;
}

static acp_status check_dec_shape(int B, int H, int C, int d, acp_dtype dt) {
    if (B <= 0 || H <= 0 || C <= 0 || d <= 0)
        return fail(ACP_EINVAL, "sizes must be positive (B=%d H=%d C=%d d=%d)", B, H, C, d);
    if (dt != ACP_F32 && dt != ACP_BF16) return fail(ACP_EINVAL, "unknown dtype %d", (int)dt);
    if (d != 64 && d != 128) return fail(ACP_EUNSUPPORTED, "head dim %d not in {64, 128}", d);
    if (C % 64 != 0 || C > 64 * 2048)
        return fail(ACP_EUNSUPPORTED, "cache size C=%d is not a multiple of 64 up to 131072", C);
    if ((long long)B * H > 65535)
        return fail(ACP_EUNSUPPORTED, "B*H=%lld exceeds 65535", (long long)B * H);
    return ACP_OK;
}

static acp_status check_state(void* state, size_t state_bytes, const DecLayout& y) {
    acp_status s = check_ptr(state, "state");
    if (s != ACP_OK) return s;
    if (state_bytes < y.total)
        return fail(ACP_EWORKSPACE, "decoding state of %zu bytes, %zu needed", state_bytes,
                    y.total);
    return ACP_OK;
}

static acp_status check_lmax(int64_t L_max) {
    if (L_max < 1 || L_max > ((int64_t)1 << 31))
        return fail(ACP_EINVAL, "L_max=%lld outside [1, 2^31]", (long long)L_max);
    return ACP_OK;
}

acp_status acp_decode_state_size(int B, int H, int C, int d, acp_dtype dt, size_t* bytes) {
    ACP_TRY(check_dec_shape(B, H, C, d, dt));
    if (bytes == nullptr) return fail(ACP_EINVAL, "bytes is NULL");
    *bytes = dec_layout(B, H, C, d, dt).total;
    return ok();
}

acp_status acp_decode_offsets(int B, int H, int C, int d, acp_dtype dt, acp_decode_layout* out) {
    ACP_TRY(check_dec_shape(B, H, C, d, dt));
    if (out == nullptr) return fail(ACP_EINVAL, "out is NULL");
    const DecLayout y = dec_layout(B, H, C, d, dt);
    out->k_cache = y.k;
    out->v_cache = y.v;
    out->c = y.c;
    out->cum = y.cum;
    out->delta = y.delta;
    out->pointer = y.ptr;
    out->flags = y.flags;
    out->total = y.total;
    return ok();
}

acp_status acp_decode_init(const void* K, const void* V, const float* log_f,
                           const float* gamma_q, const float* gamma_k, acp_dtype dt, int B,
                           int H, int L0, int C, int d, double eps, int64_t L_max, void* state,
                           size_t state_bytes, void* stream) {
    ACP_TRY(check_dec_shape(B, H, C, d, dt));
    ACP_TRY(check_eps(eps));
    ACP_TRY(check_lmax(L_max));
    if (L0 <= 0 || L0 > 64 * 2048)
        return fail(ACP_EUNSUPPORTED, "prompt length L0=%d outside [1, 131072]", L0);
    if ((int64_t)L0 > L_max) return fail(ACP_EINVAL, "L0=%d exceeds L_max=%lld", L0, (long long)L_max);
    ACP_TRY(check_ptr(K, "K"));
    ACP_TRY(check_ptr(V, "V"));
    ACP_TRY(check_ptr(log_f, "log_f"));
    ACP_TRY(check_ptr(gamma_q, "gamma_q"));
    ACP_TRY(check_ptr(gamma_k, "gamma_k"));
    const DecLayout y = dec_layout(B, H, C, d, dt);
    ACP_TRY(check_state(state, state_bytes, y));
    char* w = (char*)state;
    acp::DecodeInitArgs a{};
    a.K = K; a.V = V; a.log_f = log_f; a.gamma_q = gamma_q; a.gamma_k = gamma_k;
    a.bf16 = dt == ACP_BF16;
    a.B = B; a.H = H; a.L0 = L0; a.C = C; a.d = d;
    a.log_lmax_over_eps = eps == 0.0 ? INFINITY : std::log((double)L_max) - std::log(eps);
    a.Kc = w + y.k; a.Vc = w + y.v; a.cc = (float*)(w + y.c);
    a.cs = (double*)(w + y.cum); a.ptr = (int*)(w + y.ptr);
    a.delta = (double*)(w + y.delta); a.flags = (int*)(w + y.flags);
    return hip_status(acp::launch_decode_init(a, (hipStream_t)stream), "acp_decode_init launch");
}

acp_status fox_attn_decode(const void* q, const void* k, const void* v, const float* log_f,
                           acp_dtype dt, int B, int H, int t, int C, int d, int64_t L_max,
                           void* O, float* lse, void* state, size_t state_bytes, void* stream) {
    ACP_TRY(check_dec_shape(B, H, C, d, dt));
    ACP_TRY(check_lmax(L_max));
    if (t < 1 || (int64_t)t >= L_max)
        return fail(ACP_EINVAL, "position t=%d outside [1, L_max=%lld)", t, (long long)L_max);
    ACP_TRY(check_ptr(q, "q"));
    ACP_TRY(check_ptr(k, "k"));
    ACP_TRY(check_ptr(v, "v"));
    ACP_TRY(check_ptr(log_f, "log_f"));
    ACP_TRY(check_ptr(O, "O"));
    ACP_TRY(check_ptr(lse, "lse"));
    const DecLayout y = dec_layout(B, H, C, d, dt);
    ACP_TRY(check_state(state, state_bytes, y));
    char* w = (char*)state;
    acp::DecodeArgs a{};
    a.q = q; a.k = k; a.v = v; a.log_f = log_f; a.bf16 = dt == ACP_BF16;
    a.B = B; a.H = H; a.t = t; a.C = C; a.d = d;
    a.Kc = w + y.k; a.Vc = w + y.v; a.cc = (float*)(w + y.c);
    a.cs = (double*)(w + y.cum); a.ptr = (int*)(w + y.ptr);
    a.delta = (const double*)(w + y.delta); a.flags = (int*)(w + y.flags);
    a.part = (float*)(w + y.part);
    a.O = O; a.lse = lse;
    return hip_status(acp::launch_decode(a, (hipStream_t)stream), "fox_attn_decode launch");
}

const char* acp_status_string(acp_status s) {
    switch (s) {
        case ACP_OK: return "ok";
        case ACP_EINVAL: return "invalid argument";
        case ACP_EUNSUPPORTED: return "unsupported shape";
        case ACP_EWORKSPACE: return "workspace too small";
        case ACP_EHIP: return "HIP error";
    }
    return "unknown status";
}

const char* acp_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
