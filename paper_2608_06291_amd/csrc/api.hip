// C ABI of libbakron.so: factor handles, the divide-and-conquer schedule and
// the solve driver.  See include/bakron.h for the contract.
#include "common.h"
#include "bakron.h"

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <map>
#include <memory>
#include <mutex>
#include <set>
#include <new>
#include <functional>
#include <string>
#include <tuple>
#include <vector>

namespace bk {
using FactorOp = std::function<hipError_t()>;
void factor_ops(std::vector<FactorOp>& ops, hipStream_t s, hipStream_t s2, hipEvent_t ev_panel,
                hipEvent_t ev_rest, const float* X, int64_t d, double lam, double* Z, double* Ninv,
                double* T, double* mean, int* fail, int64_t* fail_pivot, float* packed, int64_t nt);
hipError_t pack_identity(hipStream_t s, int64_t nt, float* packed);
hipError_t unpack_factor(hipStream_t s, const float* packed, int64_t d, float* dst);

hipError_t run_plan(hipStream_t st, hipStream_t side, const Plan& plan, const float* W, int64_t m,
                    int64_t n, int mt, int nt, const Workspace& ws, const float* LA, const float* LB,
                    int b_ident, const QuantArgs& q, int8_t* codes, float* V, float* pre,
                    int knear, int spin_limit, const int4* items, hipEvent_t* tim,
                    hipEvent_t* ev_rel, hipEvent_t* ev_side);
hipError_t check_scales(hipStream_t st, const float* s, int64_t count, int* bad);
int plan_timed_launches(const Plan& plan);
hipError_t run_antidiag(hipStream_t st, const float* W, int64_t m, int64_t n, float* Wt,
                        float* delta, const float* LA, const float* LB, const QuantArgs& q,
                        int8_t* codes, float* V, float* pre);
size_t gptq_workspace_floats(int64_t m, int64_t n);
hipError_t run_gptq(hipStream_t st, const float* W, int64_t m, int64_t n, const float* LA, float* E,
                    const QuantArgs& q, int8_t* codes, float* V, float* pre, int range_tiles);
}  // namespace bk

struct bakron_factors {
    int device = 0;
    int64_t n = 0, m = 0;
    int b_ident = 0;
    float damp = 0.0f;
    float* LA = nullptr;     // packed, ceil(n/TS) tiles per side
    float* LB = nullptr;     // packed, ceil(m/TS) tiles per side (null if identity)
    int64_t LB_tiles = 0;    // tiles per side of LB storage (identity: grown on demand)
    // solve workspace (cached for the last (m, n))
    int64_t ws_m = -1, ws_n = -1;
    void* ws_mem = nullptr;         // X, Y tile arrays, flags, counters, status (bk::Workspace)
    bk::Workspace ws{};
    int knear = 8;
    // node macro tile: 0 per node (default), 4 or 2 forced (BAKRON_MACRO)
    int macro = 0;
    // BAKRON_POISON=1 at creation: fill the workspace with NaN / -1 before
    // every solve (debug aid: the solve must never read a word it did not
    // write first)
    int poison = 0;
    size_t ws_bytes = 0;
    // plan[0]: everything on the caller's stream; plan[1]: with side ops
    // (empty if the side stream is not used).  Both make the same additions
    // to every tile in the same order, so their results are identical.
    bk::Plan plan[2];
    int last_plan = 0;
    // with the cost model's choice (BAKRON_DEFER unset) a two-stream plan is
    // timed against the one-stream plan on the first solve of its shape
    int tune = 0;
    hipEvent_t tev[2] = {nullptr, nullptr};
    const int4* items = nullptr;    // device copy, owned by the process-wide plan cache
    // measurement hook: per timed launch (enqueue order) its class and work
    int prof = 0;
    int prof_valid = 0;
    std::vector<hipEvent_t> tim;
    std::vector<int> tclass[2];     // per plan: 0 prep, 1 segment, 2 node
    std::vector<double> tflops[2], tmfma[2];
    // with deferred node pushes: the side stream (CUs [side_cu_lo, #CUs)) and
    // the stream that carries the main ops (the other CUs); both forked from
    // and joined back into the caller's stream (null if not used yet)
    hipStream_t side = nullptr, main = nullptr;
    int side_cu_lo = -1;
    std::vector<hipEvent_t> ev_rel, ev_side;
    hipEvent_t ev_fork = nullptr, ev_join = nullptr;
    // set once a bakron_solve_noalloc on this handle has used its device's
    // static scratch (bakron_solve_check then reads that status word too)
    int noalloc_used = 0;
    int* noalloc_status = nullptr;   // give-up word of the last allocation-free solve
    // B = I: the one-sided (GPTQ) path and its error workspace (E rows, then
    // one int for the debug scale check); BAKRON_GPTQ=0 at creation sends
    // B = I solves through the two-sided solver instead
    int gptq = 1;
    int gptq_range = 0;   // column tiles per one-sided range (0: the library's default)
    int64_t gq_m = -1, gq_n = -1;
    float* gq_mem = nullptr;
    // BaKron-antidiagonal working copy of W and one diagonal's errors
    int64_t ad_m = -1, ad_n = -1;
    float* ad_mem = nullptr;
    std::string err;
};

static thread_local std::string g_last_error;

static const char* k_status_names[] = {"BAKRON_OK", "BAKRON_EINVAL", "BAKRON_ENOTSPD",
                                       "BAKRON_ENOMEM", "BAKRON_EHIP"};

extern "C" const char* bakron_status_string(bakron_status s) {
    int i = (int)s;
    if (i < 0 || i > 4) return "BAKRON_UNKNOWN";
    return k_status_names[i];
}

extern "C" const char* bakron_last_error(void) { return g_last_error.c_str(); }

void bk::set_last_error(const char* msg) { g_last_error = msg; }

extern "C" const char* bakron_factors_error(const bakron_factors* f) {
    return f ? f->err.c_str() : "";
}

static bakron_status hip_fail(std::string* where, hipError_t e, const char* what) {
    char buf[256];
    std::snprintf(buf, sizeof(buf), "%s: %s", what, hipGetErrorString(e));
    if (where) *where = buf;
    return (e == hipErrorOutOfMemory) ? BAKRON_ENOMEM : BAKRON_EHIP;
}

static inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Alg. 6 over tile anti-diagonals [K, L): leaf for one diagonal, otherwise
// recurse on [K, Mid), push S1 -> S2 (sources farther than knear only), then
// recurse on [Mid, L).  Split at floor((K+L)/2) (App. C: balanced splits).
static inline int imax(int a, int b) { return a > b ? a : b; }
static inline int imin(int a, int b) { return a < b ? a : b; }

// Algorithmic flops of one node launch: 2*TS^3 per (source, target) tile
// pair it pushes, mirroring the kernel's source ranges and masks.
static double node_alg_flops(int K, int Mid, int tlo, int thi, int mt, int nt, int knear,
                             int b_ident) {
    double f = 0.0;
    for (int D = tlo; D < thi; ++D) {
        for (int I = imax(0, D - (nt - 1)); I <= imin(D, mt - 1); ++I) {
            const int J = D - I;
            if (!b_ident) f += imax(0, imin(Mid - J, I - knear) - imax(K - J, 0));
            f += imax(0, imin(Mid - I, J - knear) - imax(K - I, 0));
        }
    }
    return f * 2.0 * bk::TS * bk::TS * bk::TS;
}

// Work list of a push from sources on [K, Mid) into targets on [tlo, thi)
// for MT x MT macro tiles: every (macro tile, push kind) with at least one
// target tile in [tlo, thi) and a non-empty source range, longest source
// range first.  A macro tile's source range depends only on its position, so
// a target tile receives the same sum whichever target range lists it.
static void node_items(int K, int Mid, int tlo, int thi, int mt, int nt, int knear, int b_ident,
                       int MT, std::vector<int4>& out) {
    out.clear();
    const int nmi = (mt + MT - 1) / MT, nmj = (nt + MT - 1) / MT;
    for (int mi = 0; mi < nmi; ++mi) {
        const int I0 = mi * MT;
        // macro columns whose tile anti-diagonals can meet [tlo, thi)
        const int mj_lo = imax(0, (tlo - 2 * (MT - 1) - I0 + MT - 1) / MT - 1);
        for (int mj = mj_lo; mj < nmj; ++mj) {
            const int J0 = mj * MT;
            if (I0 + J0 >= thi) break;
            bool target = false;
            for (int a = 0; a < MT && !target; ++a)
                for (int b = 0; b < MT && !target; ++b) {
                    const int I = I0 + a, J = J0 + b;
                    target = I < mt && J < nt && I + J >= tlo && I + J < thi;
                }
            if (!target) continue;
            if (!b_ident) {
                const int lo = imax(0, K - (J0 + MT - 1));
                const int hi = imin(imin(Mid - J0, I0 + MT - 1 - knear), mt);
                if (hi > lo) out.push_back(int4{I0, J0, (lo << 1) | 0, hi});
            }
            const int lo = imax(0, K - (I0 + MT - 1));
            const int hi = imin(imin(Mid - I0, J0 + MT - 1 - knear), nt);
            if (hi > lo) out.push_back(int4{I0, J0, (lo << 1) | 1, hi});
        }
    }
    std::stable_sort(out.begin(), out.end(), [](const int4& u, const int4& v) {
        return (u.w - (u.z >> 1)) > (v.w - (v.z >> 1));
    });
}

static inline int diag_lo(int D, int nt) { return imax(0, D - (nt - 1)); }
static inline int diag_hi(int D, int mt) { return imin(D, mt - 1); }

// Alg. 6 over tile anti-diagonals [K, L).  A subtree no wider than knear + 1
// anti-diagonals becomes one persistent segment launch (all its pairs are at
// distance <= knear and are pulled by their targets); a wider one recurses on
// [K, Mid), pushes S1 -> S2 for pairs farther apart than knear, then recurses
// on [Mid, L).  Split at floor((K+L)/2) (App. C: balanced splits).  With
// `defer`, a node's push is cut by the segments of its right subtree: the
// part into the first one is a main op, the others are side ops released
// after the left subtree (they may run while the segments before their
// targets are solved).
static void leaves(int K, int L, int knear, std::vector<std::pair<int, int>>& out) {
    if (L - K <= knear + 1) {
        out.push_back({K, L});
        return;
    }
    const int Mid = (K + L) / 2;
    leaves(K, Mid, knear, out);
    leaves(Mid, L, knear, out);
}

// macro: 0 chooses the macro tile per node (128 x 128 when a node has at
// least 1536 such items, three rounds of the 512 that the chip holds at
// once, else 64 x 64: with fewer, the last round of 128 x 128 items leaves
// most CUs idle); 4 or 2 forces one size
static bool node_op(int K, int Mid, int tlo, int thi, int mt, int nt, int knear, int b_ident,
                    std::vector<int4>& items, bk::PlanOp& op, int macro) {
    const double T = bk::TS;
    int MT = macro == 2 ? 2 : bk::MACRO;
    std::vector<int4> its;
    node_items(K, Mid, tlo, thi, mt, nt, knear, b_ident, MT, its);
    if (macro == 0 && (int)its.size() < 1536) {
        MT = 2;
        node_items(K, Mid, tlo, thi, mt, nt, knear, b_ident, 2, its);
    }
    if (its.empty()) return false;
    op = bk::PlanOp{};
    op.kind = 1;
    op.K = K;
    op.Mid = Mid;
    op.L = thi;
    op.tlo = tlo;
    op.thi = thi;
    op.macro = MT;
    op.item_off = (int)items.size();
    op.item_cnt = (int)its.size();
    op.rel = -1;
    const double chunkf = 2.0 * (MT * T) * (MT * T) * T;
    for (const int4& it : its) op.mfma_flops += (it.w - (it.z >> 1)) * chunkf;
    op.flops = node_alg_flops(K, Mid, tlo, thi, mt, nt, knear, b_ident);
    items.insert(items.end(), its.begin(), its.end());
    return true;
}

static void build_ops(int K, int L, int mt, int nt, int knear, int b_ident, bool defer,
                      bk::Plan& plan, std::vector<int4>& items, int macro) {
    const double T = bk::TS, pair = 2.0 * T * T * T;
    if (L - K <= knear + 1) {
        bk::PlanOp op{};
        op.kind = 0;
        op.K = K;
        op.L = L;
        double pulls = 0.0;
        int total = 0;
        for (int D = K; D < L; ++D)
            for (int I = diag_lo(D, nt); I <= diag_hi(D, mt); ++I) {
                const int J = D - I;
                ++total;
                if (!b_ident) pulls += imin(I, knear);
                pulls += imin(J, knear);
            }
        op.Mid = K;
        op.tlo = K;
        op.thi = L;
        op.rel = -1;
        op.strip_lo = imax(0, K - (mt - 1));
        op.nstrips = imin(nt - 1, L - 1) - op.strip_lo + 1;
        op.counter = plan.nseg++;
        op.flops = total * 2.0 * T * T * (T - 1.0) + pulls * pair;   // in-tile pairs + pulls
        op.mfma_flops = pulls * pair;
        plan.ops.push_back(op);
        return;
    }
    const int Mid = (K + L) / 2;
    build_ops(K, Mid, mt, nt, knear, b_ident, defer, plan, items, macro);
    // With `defer`, the push into the first right segment is a main op and the
    // pushes into the later segments are side ops released after the left
    // subtree; every target tile receives one addition per node either way.
    const int rel = (int)plan.ops.size() - 1;
    std::vector<std::pair<int, int>> right;
    leaves(Mid, L, knear, right);
    bk::PlanOp op;
    if (node_op(K, Mid, Mid, defer ? right[0].second : L, mt, nt, knear, b_ident, items, op, macro))
        plan.ops.push_back(op);
    if (defer)
        for (size_t j = 1; j < right.size(); ++j)
            if (node_op(K, Mid, right[j].first, right[j].second, mt, nt, knear, b_ident, items, op,
                        macro)) {
                op.rel = rel;
                plan.side.push_back(op);
            }
    build_ops(Mid, L, mt, nt, knear, b_ident, defer, plan, items, macro);
}

// side ops in deadline order (target segment, then release); per main op the
// number of side ops that must be complete before it (those whose targets
// start at or before its own); the host enqueue order
static void finish_plan(bk::Plan& plan) {
    std::stable_sort(plan.side.begin(), plan.side.end(), [](const bk::PlanOp& a, const bk::PlanOp& b) {
        return a.tlo != b.tlo ? a.tlo < b.tlo : a.rel < b.rel;
    });
    for (bk::PlanOp& op : plan.ops) op.rec_rel = 0;
    for (const bk::PlanOp& so : plan.side) plan.ops[so.rel].rec_rel = 1;
    size_t c = 0;
    for (bk::PlanOp& op : plan.ops) {
        while (c < plan.side.size() && plan.side[c].tlo <= op.tlo) ++c;
        op.need_side = (int)c;
    }
    plan.order.clear();
    size_t ps = 0;
    for (size_t i = 0; i < plan.ops.size(); ++i) {
        plan.order.push_back({0, (int)i});
        while (ps < plan.side.size() && plan.side[ps].rel <= (int)i) plan.order.push_back({1, (int)ps++});
    }
}

static void build_plan(int mt, int nt, int knear, int b_ident, bool defer, bk::Plan& plan,
                       std::vector<int4>& items, int macro = 0) {
    plan.ops.clear();
    plan.side.clear();
    plan.nseg = 0;
    items.clear();
    build_ops(0, mt + nt - 1, mt, nt, knear, b_ident, defer, plan, items, macro);
    finish_plan(plan);
}

extern "C" bakron_status bakron_factor(const float* A, int64_t n, const float* B, int64_t m,
                                      float damp, hipStream_t stream, bakron_factors** out) {
    g_last_error.clear();
    if (!A || n <= 0 || !out || (B && m <= 0) || !(damp >= 0.0f) || !std::isfinite(damp)) {
        g_last_error = "bakron_factor: invalid argument";
        return BAKRON_EINVAL;
    }
    if (n > (int64_t)1 << 20 || (B && m > (int64_t)1 << 20)) {
        g_last_error = "bakron_factor: dimension too large";
        return BAKRON_EINVAL;
    }
    bakron_factors* f = new (std::nothrow) bakron_factors();
    if (!f) return BAKRON_ENOMEM;
    hipGetDevice(&f->device);
    f->n = n;
    f->m = B ? m : 0;
    f->b_ident = B ? 0 : 1;
    f->damp = damp;
    if (const char* pz = std::getenv("BAKRON_POISON")) f->poison = std::atoi(pz) != 0;
    if (const char* kn = std::getenv("BAKRON_KNEAR")) {
        int v = std::atoi(kn);
        if (v >= 0 && v <= bk::KNEAR_MAX) f->knear = v;
    }
    if (const char* gq = std::getenv("BAKRON_GPTQ")) f->gptq = std::atoi(gq) != 0;
    if (const char* gr = std::getenv("BAKRON_GPTQ_RANGE")) {
        const int v = std::atoi(gr);
        if (v >= 1 && v <= 64) f->gptq_range = v;
    }
    if (const char* mc = std::getenv("BAKRON_MACRO")) {
        int v = std::atoi(mc);
        if (v == 2 || v == 4) f->macro = v;
    }

    // A and B are factored concurrently (their block steps are latency-bound):
    // B on a second, non-blocking stream forked from and joined back into
    // `stream`, each with its own scratch; each factorisation has one more
    // stream for the trailing updates it runs one panel ahead of (d >= 8192)
    const int64_t ntA = cdiv(n, bk::TS);
    double *Z[2] = {nullptr, nullptr}, *Ninv[2] = {nullptr, nullptr}, *T[2] = {nullptr, nullptr};
    double* scal = nullptr;
    int* flags = nullptr;
    hipStream_t sB = nullptr;
    hipEvent_t ev[2] = {nullptr, nullptr};
    hipStream_t s2[2] = {nullptr, nullptr};
    hipEvent_t evp[2] = {nullptr, nullptr}, evr[2] = {nullptr, nullptr};
    bakron_status st = BAKRON_OK;
    hipError_t e = hipSuccess;
    auto cleanup = [&]() {
        for (int k = 0; k < 2; ++k) {
            if (Z[k]) hipFree(Z[k]);
            if (Ninv[k]) hipFree(Ninv[k]);
            if (T[k]) hipFree(T[k]);
            if (ev[k]) hipEventDestroy(ev[k]);
            if (evp[k]) hipEventDestroy(evp[k]);
            if (evr[k]) hipEventDestroy(evr[k]);
            if (s2[k]) hipStreamDestroy(s2[k]);
        }
        if (scal) hipFree(scal);
        if (flags) hipFree(flags);
        if (sB) hipStreamDestroy(sB);
    };
    for (int k = 0; k < (B ? 2 : 1) && e == hipSuccess; ++k) {
        const size_t d = (size_t)(k == 0 ? n : m);
        const size_t zbytes = sizeof(double) * d * d;
        const size_t tbytes = sizeof(double) * (d * d / 4 + d * 64 + 64 * 64 + 64);
        if ((e = hipMalloc(&Z[k], zbytes)) == hipSuccess && (e = hipMalloc(&Ninv[k], zbytes)) == hipSuccess)
            e = hipMalloc(&T[k], tbytes);
    }
    if (e == hipSuccess) e = hipMalloc(&scal, 4 * sizeof(double));
    if (e == hipSuccess) e = hipMalloc(&flags, 8 * sizeof(int64_t));
    if (e != hipSuccess) {
        st = hip_fail(&g_last_error, e, "bakron_factor: hipMalloc (factor scratch)");
        cleanup();
        delete f;
        return st;
    }
    e = hipMemsetAsync(flags, 0, 8 * sizeof(int64_t), stream);
    // the look-ahead pays only where a trailing update outlasts the next
    // panel's chain of small launches; smaller factors create no stream
    for (int k = 0; k < (B ? 2 : 1) && e == hipSuccess; ++k) {
        if ((k == 0 ? n : m) < 8192) continue;
        e = hipStreamCreateWithFlags(&s2[k], hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&evp[k], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&evr[k], hipEventDisableTiming);
    }
    if (e == hipSuccess && B) {
        e = hipStreamCreateWithFlags(&sB, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&ev[0], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&ev[1], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventRecord(ev[0], stream);
        if (e == hipSuccess) e = hipStreamWaitEvent(sB, ev[0], 0);
    }
    if (e == hipSuccess)
        e = hipMalloc(&f->LA, sizeof(float) * (size_t)(ntA * (ntA + 1) / 2) * bk::TILE_ELEMS);
    if (e == hipSuccess && B) {
        const int64_t mtB = cdiv(m, bk::TS);
        f->LB_tiles = mtB;
        e = hipMalloc(&f->LB, sizeof(float) * (size_t)(mtB * (mtB + 1) / 2) * bk::TILE_ELEMS);
    }
    // the two factorisations' enqueue steps, interleaved so that both streams
    // start at once
    std::vector<bk::FactorOp> opsA, opsB;
    if (e == hipSuccess && B)
        bk::factor_ops(opsB, sB, s2[1], evp[1], evr[1], B, m, (double)damp, Z[1], Ninv[1], T[1],
                       scal + 1, flags + 1, reinterpret_cast<int64_t*>(flags) + 3, f->LB, f->LB_tiles);
    if (e == hipSuccess)
        bk::factor_ops(opsA, stream, s2[0], evp[0], evr[0], A, n, (double)damp, Z[0], Ninv[0], T[0],
                       scal, flags, reinterpret_cast<int64_t*>(flags) + 2, f->LA, ntA);
    for (size_t i = 0; e == hipSuccess && (i < opsA.size() || i < opsB.size()); ++i) {
        if (i < opsB.size()) e = opsB[i]();
        if (e == hipSuccess && i < opsA.size()) e = opsA[i]();
    }
    if (e == hipSuccess && B) {
        e = hipEventRecord(ev[1], sB);
        if (e == hipSuccess) e = hipStreamWaitEvent(stream, ev[1], 0);
    }
    if (e != hipSuccess) {
        st = hip_fail(&g_last_error, e, "bakron_factor: launch");
        if (sB) (void)hipStreamSynchronize(sB);
        for (hipStream_t x : s2)
            if (x) (void)hipStreamSynchronize(x);
        cleanup();
        bakron_factors_free(f);
        return st;
    }
    int64_t hflags[8];
    e = hipMemcpyAsync(hflags, flags, sizeof(hflags), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    cleanup();
    if (e != hipSuccess) {
        st = hip_fail(&g_last_error, e, "bakron_factor: synchronize");
        bakron_factors_free(f);
        return st;
    }
    const int* hf = reinterpret_cast<const int*>(hflags);
    for (int which = 0; which < 2; ++which) {
        if (hf[which]) {
            const int64_t d = which == 0 ? n : m;
            const int64_t piv = hflags[2 + which];
            char buf[200];
            std::snprintf(buf, sizeof(buf),
                          "bakron_factor: damped %s is not positive definite (pivot %lld of RevCholesky, "
                          "original index %lld)",
                          which == 0 ? "A" : "B", (long long)piv, (long long)(d - 1 - piv));
            g_last_error = buf;
            bakron_factors_free(f);
            return BAKRON_ENOTSPD;
        }
    }
    *out = f;
    return BAKRON_OK;
}

extern "C" void bakron_factors_free(bakron_factors* f) {
    if (!f) return;
    int cur = 0;
    hipGetDevice(&cur);
    if (cur != f->device) hipSetDevice(f->device);
    hipDeviceSynchronize();
    if (f->LA) hipFree(f->LA);
    if (f->LB) hipFree(f->LB);
    if (f->ws_mem) hipFree(f->ws_mem);
    if (f->ad_mem) hipFree(f->ad_mem);
    if (f->gq_mem) hipFree(f->gq_mem);
    // f->side, f->main and f->items belong to the process-wide plan cache
    for (hipEvent_t ev : f->tev)
        if (ev) hipEventDestroy(ev);
    if (f->ev_fork) hipEventDestroy(f->ev_fork);
    if (f->ev_join) hipEventDestroy(f->ev_join);
    for (hipEvent_t ev : f->ev_rel) hipEventDestroy(ev);
    for (hipEvent_t ev : f->ev_side) hipEventDestroy(ev);
    for (hipEvent_t ev : f->tim) hipEventDestroy(ev);
    if (cur != f->device) hipSetDevice(cur);
    delete f;
}

// B = I: the packed identity factor grows to the requested m
static bakron_status ensure_identity(bakron_factors* f, int64_t mt) {
    if (!f->b_ident || f->LB_tiles >= mt) return BAKRON_OK;
    if (f->LB) hipFree(f->LB);
    f->LB = nullptr;
    hipError_t e = hipMalloc(&f->LB, sizeof(float) * (size_t)(mt * (mt + 1) / 2) * bk::TILE_ELEMS);
    if (e == hipSuccess) e = bk::pack_identity(0, mt, f->LB);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: identity factor");
    f->LB_tiles = mt;
    return BAKRON_OK;
}

// The plan of an mt x nt tile grid.  Node pushes into later segments go to a
// side stream restricted to the CUs that no segment launch needs (a segment
// has one persistent workgroup per strip, at most one per CU): CUs
// [R, #CUs) with R = max(#CUs / 2, widest segment rounded up to 32), when at
// least 64 CUs remain.  BAKRON_DEFER=0 keeps every push on the caller's
// stream, and so does a failure to create the side stream.
// Launch plans, their node work lists on the device and the two CU-restricted
// streams depend only on the device and the solve shape, so they are built
// once per process and shared by every handle (read-only; kept until the
// process ends).  Handles that fork onto the same streams concurrently are
// serialised on them, which keeps each solve's ordering intact.
struct PlanEntry {
    bk::Plan plan[2];
    const int4* items = nullptr;
    hipStream_t main = nullptr, side = nullptr;
};
static std::mutex g_plan_mu;
static std::map<std::tuple<int, int, int, int, int, int, int>, std::shared_ptr<PlanEntry>> g_plans;
static std::map<std::pair<int, int>, std::pair<hipStream_t, hipStream_t>> g_streams;
static std::set<int> g_streams_tried;   // devices whose default stream pair was requested

// At process exit (registered once, after the HIP runtime has initialised, so
// it runs before the runtime's own teardown): destroy the cached streams and
// free the device work lists, so that no CU-restricted queue outlives the
// program's last call.
static void release_plan_cache() {
    std::lock_guard<std::mutex> lock(g_plan_mu);
    for (auto& kv : g_streams) {
        (void)hipStreamDestroy(kv.second.first);
        (void)hipStreamDestroy(kv.second.second);
    }
    g_streams.clear();
    for (auto& kv : g_plans)
        if (kv.second->items) (void)hipFree(const_cast<int4*>(kv.second->items));
    g_plans.clear();
    (void)hipGetLastError();
}

static void register_release() {
    static const bool registered = std::atexit(release_plan_cache) == 0;
    (void)registered;
}

// main ops on CUs [0, R), side ops on [R, #CUs): a persistent segment
// workgroup never sits on a CU a side push waits for, and the reverse
static bool masked_streams(int device, int ncu, int R, hipStream_t* main, hipStream_t* side) {
    auto it = g_streams.find({device, R});
    if (it != g_streams.end()) {
        *main = it->second.first;
        *side = it->second.second;
        return true;
    }
    auto masked = [&](int lo, int hi, hipStream_t* out) {
        std::vector<uint32_t> mask((size_t)(ncu + 31) / 32, 0u);
        for (int c = lo; c < hi; ++c) mask[(size_t)c / 32] |= 1u << (c % 32);
        if (hipExtStreamCreateWithCUMask(out, (uint32_t)mask.size(), mask.data()) != hipSuccess ||
            !*out) {
            *out = nullptr;
            (void)hipGetLastError();
            return false;
        }
        return true;
    };
    hipStream_t m = nullptr, sd = nullptr;
    if (!masked(0, R, &m) || !masked(R, ncu, &sd)) {
        if (m) (void)hipStreamDestroy(m);
        return false;
    }
    g_streams[{device, R}] = {m, sd};
    register_release();
    *main = m;
    *side = sd;
    return true;
}

// Modelled duration of a plan (seconds): main ops in order, side ops in
// order, a side op starting after the main op it is released by, a main op
// after the side ops it waits for, each wait across the two streams adding
// a fixed latency.  A segment costs a fixed time per tile anti-diagonal (its
// sequential chain); a node push a fixed launch cost plus its MFMA flops at
// a per-CU rate on the CUs of its stream, a side push a larger fixed cost.
// The constants are fitted to MI355X solve times of twelve layer shapes
// (3072^2 to 14336 x 4096) under both plans; only the comparison of the two
// plans for one shape uses them.
static double plan_model_seconds(const bk::Plan& p, int cus_main, int cus_side) {
    const double t_diag = 13.4e-6, t_seg = 3e-6, t_node = 6e-6, t_side = 30e-6, t_wait = 40e-6;
    const double rate_cu = 0.45e12;
    std::vector<double> main_end(p.ops.size(), 0.0), side_end(p.side.size(), 0.0);
    double tm = 0.0, ts = 0.0;
    size_t next_side = 0;
    auto run_side = [&](size_t upto) {
        for (; next_side < upto; ++next_side) {
            const bk::PlanOp& o = p.side[next_side];
            ts = std::max(ts, main_end[o.rel] + t_wait) + t_side +
                 o.mfma_flops / (rate_cu * cus_side);
            side_end[next_side] = ts;
        }
    };
    for (size_t i = 0; i < p.ops.size(); ++i) {
        const bk::PlanOp& o = p.ops[i];
        run_side((size_t)o.need_side);
        if (o.need_side > 0) tm = std::max(tm, side_end[o.need_side - 1] + t_wait);
        tm += o.kind == 0 ? t_seg + (o.L - o.K) * t_diag
                          : t_node + o.mfma_flops / (rate_cu * cus_main);
        main_end[i] = tm;
    }
    run_side(p.side.size());
    return std::max(tm, ts);
}

// first CU of the side stream on a device with ncu CUs (the main stream
// keeps at least half of them and one CU per strip of the widest segment),
// or 0 when fewer than 64 CUs would be left for the side stream
static int side_split(const bk::Plan& one, int ncu) {
    int widest = 0;
    for (const bk::PlanOp& op : one.ops)
        if (op.kind == 0) widest = imax(widest, op.nstrips);
    const int R = imax(ncu / 2, (widest + 31) / 32 * 32);
    return (ncu > 0 && ncu - R >= 64) ? R : 0;
}

// defer: 0 never, 1 whenever enough CUs are free, 2 when the modelled
// duration of the two-stream plan is below that of the one-stream plan
static bool use_two_streams(const bk::Plan& one, const bk::Plan& two, int R, int ncu, int defer) {
    if (R <= 0 || two.side.empty() || defer == 0) return false;
    // the overlap pays only while the pushes into later segments fit on
    // the side CUs during the chain; with more push work (tall or wide
    // layers) one stream with every CU per push is faster
    return defer == 1 || plan_model_seconds(two, R, ncu - R) < plan_model_seconds(one, ncu, 0);
}

static bakron_status build_plan_entry(bakron_factors* f, int mt, int nt, int defer,
                                      PlanEntry& pe) {
    std::vector<int4> items_host;
    build_plan(mt, nt, f->knear, f->b_ident, false, pe.plan[0], items_host, f->macro);
    pe.plan[1] = bk::Plan{};
    int ncu = 0;
    hipDeviceProp_t prop;
    if (defer && hipGetDeviceProperties(&prop, f->device) == hipSuccess) ncu = prop.multiProcessorCount;
    const int R = side_split(pe.plan[0], ncu);
    if (R > 0) {
        bk::Plan deferred;
        std::vector<int4> items;
        build_plan(mt, nt, f->knear, f->b_ident, true, deferred, items, f->macro);
        deferred.side_cu_lo = R;
        const bool use = use_two_streams(pe.plan[0], deferred, R, ncu, defer);
        if (use && masked_streams(f->device, ncu, R, &pe.main, &pe.side)) {
            const int off = (int)items_host.size();
            for (bk::PlanOp& op : deferred.ops) if (op.kind == 1) op.item_off += off;
            for (bk::PlanOp& op : deferred.side) op.item_off += off;
            items_host.insert(items_host.end(), items.begin(), items.end());
            pe.plan[1] = std::move(deferred);
        }
    }
    if (!items_host.empty()) {
        int4* dev = nullptr;
        const size_t ib = sizeof(int4) * items_host.size();
        hipError_t e = hipMalloc(&dev, ib);
        if (e == hipSuccess) e = hipMemcpy(dev, items_host.data(), ib, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            if (dev) hipFree(dev);
            return hip_fail(&f->err, e, "bakron_solve: work list upload");
        }
        pe.items = dev;
    }
    return BAKRON_OK;
}

static bakron_status plan_with_side_stream(bakron_factors* f, int mt, int nt) {
    const char* env = std::getenv("BAKRON_DEFER");
    const int defer = env ? (std::atoi(env) == 0 ? 0 : 1) : 2;
    const auto key = std::make_tuple(f->device, mt, nt, f->knear, f->b_ident, defer, f->macro);
    std::shared_ptr<PlanEntry> pe;
    {
        std::lock_guard<std::mutex> lock(g_plan_mu);
        // The default pair of CU-restricted streams (main on half the CUs) is
        // created at the first solve planned on a device, whichever plan that
        // shape uses: created only after one-stream solves had run on the
        // caller's stream, they made later two-stream solves about 25% slower
        // on MI355X (4096 x 4096: 6.0 ms against 4.7 ms).
        if (defer != 0 && !g_streams_tried.count(f->device)) {
            g_streams_tried.insert(f->device);
            hipDeviceProp_t prop;
            if (hipGetDeviceProperties(&prop, f->device) == hipSuccess) {
                const int ncu = prop.multiProcessorCount, R = ncu / 2;
                hipStream_t a = nullptr, b = nullptr;
                if (ncu - R >= 64) (void)masked_streams(f->device, ncu, R, &a, &b);
            }
        }
        auto it = g_plans.find(key);
        if (it != g_plans.end()) {
            pe = it->second;
        } else {
            pe = std::make_shared<PlanEntry>();
            bakron_status st = build_plan_entry(f, mt, nt, defer, *pe);
            if (st != BAKRON_OK) return st;
            register_release();
            g_plans[key] = pe;
        }
    }
    f->plan[0] = pe->plan[0];
    f->plan[1] = pe->plan[1];
    f->items = pe->items;
    f->main = pe->main;
    f->side = pe->side;
    f->side_cu_lo = pe->plan[1].side.empty() ? -1 : pe->plan[1].side_cu_lo;
    f->tune = defer == 2 && !pe->plan[1].side.empty();
    if (pe->plan[1].side.empty()) return BAKRON_OK;
    auto grow = [](std::vector<hipEvent_t>& v, size_t need) {
        while (v.size() < need) {
            hipEvent_t ev;
            if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) return false;
            v.push_back(ev);
        }
        return true;
    };
    if ((!f->ev_fork && hipEventCreateWithFlags(&f->ev_fork, hipEventDisableTiming) != hipSuccess) ||
        (!f->ev_join && hipEventCreateWithFlags(&f->ev_join, hipEventDisableTiming) != hipSuccess) ||
        !grow(f->ev_rel, f->plan[1].ops.size()) || !grow(f->ev_side, f->plan[1].side.size())) {
        (void)hipGetLastError();
        f->plan[1] = bk::Plan{};   // no events: every push stays on the caller's stream
    }
    return BAKRON_OK;
}

static bakron_status ensure_workspace(bakron_factors* f, int64_t m, int64_t n) {
    if (f->ws_m == m && f->ws_n == n && f->ws_mem) return BAKRON_OK;
    bakron_status st;
    const int64_t mt = cdiv(m, bk::TS), nt = cdiv(n, bk::TS);
    if (f->ws_mem) { hipFree(f->ws_mem); f->ws_mem = nullptr; }
    f->ws_m = f->ws_n = -1;
    st = plan_with_side_stream(f, (int)mt, (int)nt);
    if (st != BAKRON_OK) return st;
    const size_t tiles = (size_t)mt * (size_t)nt;
    const size_t fbytes = sizeof(float) * tiles * bk::TILE_ELEMS;
    const size_t ibytes = sizeof(int) * (tiles + (size_t)f->plan[0].nseg + 2);
    hipError_t e = hipMalloc(&f->ws_mem, 2 * fbytes + ibytes);
    if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: hipMalloc (workspace)");
    f->ws_bytes = 2 * fbytes + ibytes;
    char* base = static_cast<char*>(f->ws_mem);
    int* ints = reinterpret_cast<int*>(base + 2 * fbytes);
    int* st_words = ints + tiles + f->plan[0].nseg;   // status, scale_bad: the last two words
    f->ws = bk::Workspace{reinterpret_cast<float*>(base), reinterpret_cast<float*>(base + fbytes),
                          ints, ints + tiles, st_words, st_words + 1};
    // the give-up status is cleared here and by bakron_solve_check only
    e = hipMemset(st_words, 0, 2 * sizeof(int));
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: workspace status init");
    st = ensure_identity(f, mt);
    if (st != BAKRON_OK) return st;
    // per timed launch: class and work, in plan order
    for (int pi = 0; pi < 2; ++pi) {
        const bk::Plan& pl = f->plan[pi];
        f->tclass[pi].assign(1, 0);
        f->tflops[pi].assign(1, (double)m * n * 4.0 + 2.0 * (double)fbytes);   // bytes for class 0
        f->tmfma[pi].assign(1, 0.0);
        for (const std::pair<int, int>& o : pl.order) {
            const bk::PlanOp& op = o.first == 0 ? pl.ops[o.second] : pl.side[o.second];
            f->tclass[pi].push_back(op.kind == 0 ? 1 : 2);
            f->tflops[pi].push_back(op.flops);
            f->tmfma[pi].push_back(op.mfma_flops);
        }
    }
    f->ws_m = m;
    f->ws_n = n;
    return BAKRON_OK;
}

// the kernels' view of a quantiser (alphabet bounds, scale lookup)
static bk::QuantArgs quant_args(const bakron_quantizer& q, int64_t n) {
    bk::QuantArgs a;
    a.scale = q.scale;
    a.col_scale = q.col_scale;
    a.gsize = q.group_size;
    a.ngroups = q.group_size > 0 ? (int)cdiv(n, q.group_size) : 1;
    const int h = 1 << (q.bits - 1);
    a.qlo = q.alphabet == BAKRON_ALPHABET_ASYMMETRIC ? (float)-h : (float)-(h - 1);
    a.qhi = (float)(h - 1);
    return a;
}

// argument checks shared by the solve entry points (host side, synchronous)
static bakron_status check_solve_args(bakron_factors* f, const char* who, const float* W, int64_t m,
                                      int64_t n, bakron_quantizer q, const int8_t* codes,
                                      const float* V) {
    if (!W || !codes || !V || !q.scale || m <= 0 || n <= 0) {
        f->err = std::string(who) + ": null pointer or non-positive size";
        return BAKRON_EINVAL;
    }
    if (n != f->n || (!f->b_ident && m != f->m)) {
        f->err = std::string(who) + ": (m, n) does not match the factor handle";
        return BAKRON_EINVAL;
    }
    if (q.bits < 2 || q.bits > 8) {
        f->err = std::string(who) + ": bits must be in [2, 8]";
        return BAKRON_EINVAL;
    }
    if (q.alphabet != BAKRON_ALPHABET_SYMMETRIC && q.alphabet != BAKRON_ALPHABET_ASYMMETRIC) {
        f->err = std::string(who) + ": unknown alphabet";
        return BAKRON_EINVAL;
    }
    if (q.group_size < 0) {
        f->err = std::string(who) + ": group_size must be >= 0";
        return BAKRON_EINVAL;
    }
    if ((m + bk::TS) * (n + bk::TS) > ((int64_t)1 << 40)) {
        f->err = std::string(who) + ": matrix too large";
        return BAKRON_EINVAL;
    }
    return BAKRON_OK;
}

// debug mode: every scale must be finite and >= 0 (a device reduction into
// the flag word `bad_dev`, then one synchronisation of `stream`)
static bakron_status debug_scale_check(bakron_factors* f, const bakron_quantizer& q,
                                       const bk::QuantArgs& qa, int64_t m, int64_t n, int* bad_dev,
                                       hipStream_t stream) {
    const int64_t ns = m * (int64_t)qa.ngroups;
    int32_t bad = 0;
    hipError_t ce = hipMemsetAsync(bad_dev, 0, sizeof(int), stream);
    if (ce == hipSuccess) ce = bk::check_scales(stream, q.scale, ns, bad_dev);
    if (ce == hipSuccess && q.col_scale) ce = bk::check_scales(stream, q.col_scale, n, bad_dev);
    if (ce == hipSuccess) ce = hipMemcpyAsync(&bad, bad_dev, sizeof(bad), hipMemcpyDeviceToHost, stream);
    if (ce == hipSuccess) ce = hipStreamSynchronize(stream);
    if (ce != hipSuccess) return hip_fail(&f->err, ce, "bakron_solve_debug: scale check");
    if (bad) {
        f->err = "bakron_solve_debug: a scale is negative, NaN or infinite";
        return BAKRON_EINVAL;
    }
    return BAKRON_OK;
}

// B = I: the rows are independent (GPTQ with Hessian A on every row)
static bakron_status solve_gptq(bakron_factors* f, const float* W, int64_t m, int64_t n,
                                const bakron_quantizer& q, int8_t* codes, float* V, float* pre,
                                hipStream_t stream) {
    const size_t ef = bk::gptq_workspace_floats(m, n);
    if (f->gq_m != m || f->gq_n != n || !f->gq_mem) {
        if (f->gq_mem) { hipFree(f->gq_mem); f->gq_mem = nullptr; }
        f->gq_m = f->gq_n = -1;
        hipError_t e = hipMalloc(&f->gq_mem, sizeof(float) * ef + 256);
        if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: hipMalloc (one-sided workspace)");
        f->gq_m = m;
        f->gq_n = n;
    }
    const bk::QuantArgs qa = quant_args(q, n);
    int* bad_dev = reinterpret_cast<int*>(f->gq_mem + ef);
    if (pre) {
        bakron_status st = debug_scale_check(f, q, qa, m, n, bad_dev, stream);
        if (st != BAKRON_OK) return st;
    }
    hipError_t e = hipSuccess;
    if (f->poison) e = bk::fill_words(stream, f->gq_mem, (int64_t)ef, 0xFFFFFFFFu);
    if (e == hipSuccess) e = bk::run_gptq(stream, W, m, n, f->LA, f->gq_mem, qa, codes, V, pre, f->gptq_range);
    if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: launch (one-sided)");
    f->prof_valid = 0;   // the per-launch measurement hook covers the two-sided solver only
    return BAKRON_OK;
}

static bakron_status solve_impl(const float* W, int64_t m, int64_t n, const bakron_factors* fc,
                                bakron_quantizer q, int8_t* codes, float* V, float* pre,
                                hipStream_t stream) {
    bakron_factors* f = const_cast<bakron_factors*>(fc);
    if (!f) return BAKRON_EINVAL;
    f->err.clear();
    bakron_status st = check_solve_args(f, "bakron_solve", W, m, n, q, codes, V);
    if (st != BAKRON_OK) return st;
    if (f->b_ident && f->gptq) return solve_gptq(f, W, m, n, q, codes, V, pre, stream);
    const bool fresh = !(f->ws_m == m && f->ws_n == n && f->ws_mem);   // first solve of this shape
    st = ensure_workspace(f, m, n);
    if (st != BAKRON_OK) return st;
    const int mt = (int)cdiv(m, bk::TS), nt = (int)cdiv(n, bk::TS);
    const bk::QuantArgs qa = quant_args(q, n);
    if (pre) {
        st = debug_scale_check(f, q, qa, m, n, f->ws.scale_bad, stream);
        if (st != BAKRON_OK) return st;
    }
    // polls before a tile-ordering wait gives up; BAKRON_SPIN_LIMIT (read at
    // every solve) lowers it, to exercise the give-up path from the host
    int spin_limit = bk::SPIN_LIMIT;
    if (const char* sl = std::getenv("BAKRON_SPIN_LIMIT")) {
        const int v = std::atoi(sl);
        if (v >= 1 && v <= bk::SPIN_LIMIT) spin_limit = v;
    }
    // the legacy default stream synchronises implicitly with the (blocking)
    // CU-restricted streams, so calls on it use the one-stream plan
    const bool legacy = stream == nullptr || stream == hipStreamLegacy;
    // under stream capture all launches stay on the capturing stream (the
    // two-stream fork is not captured)
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (!legacy && hipStreamIsCapturing(stream, &cap) != hipSuccess) cap = hipStreamCaptureStatusNone;
    int pi = (!legacy && cap == hipStreamCaptureStatusNone && !f->plan[1].side.empty()) ? 1 : 0;
    // The first solve of a shape for which the cost model chose the two-stream
    // plan runs both plans (twice each, the second runs timed, one host
    // synchronisation) and keeps the faster one for the handle: the two-stream
    // time depends on what the process did on other streams before (up to 25%
    // slower on MI355X), the one-stream time does not.  Both plans write the
    // same outputs.  The first solve of a shape allocates anyway, so later
    // calls keep their no-allocation, no-synchronisation contract.
    const bool tune = fresh && f->tune && pi == 1 && !f->prof;
    if (fresh) f->tune = 0;
    f->last_plan = pi;
    hipEvent_t* tim = nullptr;
    f->prof_valid = 0;
    if (f->prof) {
        const size_t need = 2 * (size_t)bk::plan_timed_launches(f->plan[pi]);
        while (f->tim.size() < need) {
            hipEvent_t ev;
            hipError_t ee = hipEventCreate(&ev);
            if (ee != hipSuccess) return hip_fail(&f->err, ee, "bakron_solve: hipEventCreate");
            f->tim.push_back(ev);
        }
        tim = f->tim.data();
    }
    // one solve with plan `plan`; with side ops the main ops run on the
    // handle's CU-restricted main stream, forked from and joined back into
    // the caller's stream
    auto launch = [&](int plan) -> hipError_t {
        const bool fork = plan == 1;
        hipStream_t ms = fork ? f->main : stream;
        hipError_t e = hipSuccess;
        // poisoning spares the last two words (the sticky status and the scale flag)
        if (f->poison) e = bk::fill_words(stream, f->ws_mem, (int64_t)(f->ws_bytes / 4) - 2, 0xFFFFFFFFu);
        if (fork && e == hipSuccess) {
            e = hipEventRecord(f->ev_fork, stream);
            if (e == hipSuccess) e = hipStreamWaitEvent(ms, f->ev_fork, 0);
        }
        if (e == hipSuccess)
            e = bk::run_plan(ms, f->side, f->plan[plan], W, m, n, mt, nt, f->ws, f->LA, f->LB,
                             f->b_ident, qa, codes, V, pre, f->knear, spin_limit, f->items,
                             plan == pi ? tim : nullptr, f->ev_rel.data(), f->ev_side.data());
        if (fork && e == hipSuccess) {
            e = hipEventRecord(f->ev_join, ms);
            if (e == hipSuccess) e = hipStreamWaitEvent(stream, f->ev_join, 0);
        }
        return e;
    };
    hipError_t e = hipSuccess;
    if (tune) {
        for (hipEvent_t& ev : f->tev)
            if (!ev && e == hipSuccess) e = hipEventCreate(&ev);
        float t[2] = {0.0f, 0.0f};
        for (int rep = 0; rep < 2 && e == hipSuccess; ++rep)
            for (int plan = 0; plan <= 1 && e == hipSuccess; ++plan) {
                e = hipEventRecord(f->tev[0], stream);
                if (e == hipSuccess) e = launch(plan);
                if (e == hipSuccess) e = hipEventRecord(f->tev[1], stream);
                if (e == hipSuccess) e = hipEventSynchronize(f->tev[1]);
                if (e == hipSuccess && rep == 1) e = hipEventElapsedTime(&t[plan], f->tev[0], f->tev[1]);
            }
        if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: timing the plans");
        if (t[0] <= t[1]) {   // one stream from now on for this handle and shape
            f->plan[1] = bk::Plan{};
            pi = 0;
        }
        f->last_plan = pi;
        return BAKRON_OK;   // the outputs of the last run (two streams) are the solve's
    }
    e = launch(pi);
    if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: launch");
    f->prof_valid = f->prof;
    return BAKRON_OK;
}

extern "C" bakron_status bakron_solve(const float* W, int64_t m, int64_t n,
                                     const bakron_factors* f, bakron_quantizer q, int8_t* codes,
                                     float* V, hipStream_t stream) {
    return solve_impl(W, m, n, f, q, codes, V, nullptr, stream);
}

extern "C" bakron_status bakron_solve_debug(const float* W, int64_t m, int64_t n,
                                           const bakron_factors* f, bakron_quantizer q,
                                           int8_t* codes, float* V, float* pre,
                                           hipStream_t stream) {
    if (!pre) {
        if (f) const_cast<bakron_factors*>(f)->err = "bakron_solve_debug: pre is null";
        return BAKRON_EINVAL;
    }
    return solve_impl(W, m, n, f, q, codes, V, pre, stream);
}

extern "C" bakron_status bakron_solve_antidiag(const float* W, int64_t m, int64_t n,
                                             const bakron_factors* fc, bakron_quantizer q,
                                             int8_t* codes, float* V, float* pre,
                                             hipStream_t stream) {
    bakron_factors* f = const_cast<bakron_factors*>(fc);
    if (!f) return BAKRON_EINVAL;
    f->err.clear();
    bakron_status st = check_solve_args(f, "bakron_solve_antidiag", W, m, n, q, codes, V);
    if (st != BAKRON_OK) return st;
    if (m > (int64_t)1 << 30 || n > (int64_t)1 << 30) {
        f->err = "bakron_solve_antidiag: dimension too large";
        return BAKRON_EINVAL;
    }
    st = ensure_identity(f, cdiv(m, bk::TS));
    if (st != BAKRON_OK) return st;
    if (f->ad_m != m || f->ad_n != n || !f->ad_mem) {
        if (f->ad_mem) { hipFree(f->ad_mem); f->ad_mem = nullptr; }
        f->ad_m = f->ad_n = -1;
        const size_t elems = (size_t)cdiv(m * n, 64) * 64 + (size_t)(cdiv(m, bk::TS) * bk::TS);
        hipError_t e = hipMalloc(&f->ad_mem, sizeof(float) * elems);
        if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve_antidiag: hipMalloc (workspace)");
        f->ad_m = m;
        f->ad_n = n;
    }
    if (f->poison) {
        const size_t elems = (size_t)cdiv(m * n, 64) * 64 + (size_t)(cdiv(m, bk::TS) * bk::TS);
        hipError_t pe = bk::fill_words(stream, f->ad_mem, (int64_t)elems, 0xFFFFFFFFu);
        if (pe != hipSuccess) return hip_fail(&f->err, pe, "bakron_solve_antidiag: poison");
    }
    hipError_t e = bk::run_antidiag(stream, W, m, n, f->ad_mem, f->ad_mem + (size_t)cdiv(m * n, 64) * 64, f->LA,
                                    f->LB, quant_args(q, n), codes, V, pre);
    if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve_antidiag: launch");
    return BAKRON_OK;
}

extern "C" bakron_status bakron_factor_export(const bakron_factors* f, int which, float* dst,
                                             hipStream_t stream) {
    if (!f || !dst || (which != 0 && which != 1)) return BAKRON_EINVAL;
    if (which == 1 && (f->b_ident || !f->LB)) return BAKRON_EINVAL;
    const int64_t d = which == 0 ? f->n : f->m;
    hipError_t e = bk::unpack_factor(stream, which == 0 ? f->LA : f->LB, d, dst);
    if (e != hipSuccess)
        return hip_fail(&const_cast<bakron_factors*>(f)->err, e, "bakron_factor_export");
    return BAKRON_OK;
}

extern "C" bakron_status bakron_profile_enable(bakron_factors* f, int on) {
    if (!f) return BAKRON_EINVAL;
    f->prof = on ? 1 : 0;
    f->prof_valid = 0;
    return BAKRON_OK;
}

extern "C" bakron_status bakron_profile_read(const bakron_factors* f, bakron_kernel_stat* stats,
                                            int nstats) {
    if (!f || !stats || nstats < 1) return BAKRON_EINVAL;
    if (!f->prof_valid) return BAKRON_EINVAL;
    for (int k = 0; k < nstats; ++k) stats[k] = bakron_kernel_stat{0.0, 0, 0.0, 0.0};
    const int pi = f->last_plan;
    for (size_t i = 0; i < f->tclass[pi].size(); ++i) {
        float ms = 0.0f;
        hipError_t e = hipEventElapsedTime(&ms, f->tim[2 * i], f->tim[2 * i + 1]);
        if (e != hipSuccess)
            return hip_fail(&const_cast<bakron_factors*>(f)->err, e, "bakron_profile_read");
        const int k = f->tclass[pi][i];
        if (k >= nstats) continue;
        stats[k].ms += ms;
        stats[k].launches += 1;
        stats[k].flops += f->tflops[pi][i];
        stats[k].mfma_flops += f->tmfma[pi][i];
    }
    return BAKRON_OK;
}

// ---------------------------------------------------------------------------
// Allocation-free solve.  The solve workspace (the X and Y tile arrays, the
// tile ready flags, the ticket counters, the sticky give-up word) and the node
// work list live in one static device array per GPU instead of a hipMalloc'd
// buffer.  Its device address is taken once per device with
// hipGetSymbolAddress (the array's name is only a host-side stand-in) and kept
// in g_noalloc_ptr.  Plans are built on the host and cached per shape (host
// memory only); the work list is copied into the array by every call.
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)136 << 20;
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

struct HostPlan {
    bk::Plan plan;
    std::vector<int4> items;
};
static std::mutex g_noalloc_mu;
static std::map<int, unsigned char*> g_noalloc_ptr;   // device -> address of `scratch`
static std::map<std::tuple<int, int, int, int, int>, std::shared_ptr<HostPlan>> g_host_plans;

// Byte layout of the scratch array: the sticky give-up word and the scale
// flag at offset 0 (the same place for every shape), then X, Y, the ready
// flags and ticket counters, then the work list.
struct NoallocLayout {
    size_t x_off, fbytes, ints_off, items_off, total;
};
static NoallocLayout noalloc_layout(int64_t tiles, int nseg, size_t nitems) {
    NoallocLayout L;
    L.x_off = 256;
    L.fbytes = sizeof(float) * (size_t)tiles * bk::TILE_ELEMS;
    L.ints_off = L.x_off + 2 * L.fbytes;
    const size_t ibytes = sizeof(int) * ((size_t)tiles + (size_t)nseg);
    L.items_off = (L.ints_off + ibytes + 255) / 256 * 256;
    L.total = L.items_off + sizeof(int4) * nitems;
    return L;
}

extern "C" bakron_status bakron_solve_noalloc(const float* W, int64_t m, int64_t n,
                                             const bakron_factors* fc, bakron_quantizer q,
                                             int8_t* codes, float* V, hipStream_t stream) {
    bakron_factors* f = const_cast<bakron_factors*>(fc);
    if (!f) return BAKRON_EINVAL;
    f->err.clear();
    bakron_status st = check_solve_args(f, "bakron_solve_noalloc", W, m, n, q, codes, V);
    if (st != BAKRON_OK) return st;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve_noalloc: hipGetDevice");
    if (dev != f->device) {
        f->err = "bakron_solve_noalloc: the current device is not the handle's device";
        return BAKRON_EINVAL;
    }
    const int mt = (int)cdiv(m, bk::TS), nt = (int)cdiv(n, bk::TS);
    const int64_t tiles = (int64_t)mt * nt;
    // the workspace alone must fit before any plan is built
    if (256 + 2 * sizeof(float) * (size_t)tiles * bk::TILE_ELEMS > NOALLOC_SCRATCH_BYTES) {
        f->err = "bakron_solve_noalloc: layer too large for the static scratch (at most 136 MiB: "
                 "ceil(m/32) * ceil(n/32) <= 17000 tiles, e.g. 4096 x 4096)";
        return BAKRON_EINVAL;
    }
    std::shared_ptr<HostPlan> hp;
    unsigned char* base = nullptr;
    bool first_on_device = false;
    {
        std::lock_guard<std::mutex> lock(g_noalloc_mu);
        const auto key = std::make_tuple(mt, nt, f->knear, f->b_ident, f->macro);
        auto it = g_host_plans.find(key);
        if (it != g_host_plans.end()) {
            hp = it->second;
        } else {
            hp = std::make_shared<HostPlan>();
            build_plan(mt, nt, f->knear, f->b_ident, false, hp->plan, hp->items, f->macro);
            g_host_plans[key] = hp;
        }
        auto pit = g_noalloc_ptr.find(dev);
        if (pit != g_noalloc_ptr.end()) {
            base = pit->second;
        } else {
            void* ptr = nullptr;
            e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
            if (e != hipSuccess || !ptr)
                return hip_fail(&f->err, e != hipSuccess ? e : hipErrorInvalidSymbol,
                                "bakron_solve_noalloc: hipGetSymbolAddress(scratch)");
            base = static_cast<unsigned char*>(ptr);
            g_noalloc_ptr[dev] = base;
            first_on_device = true;
        }
    }
    const NoallocLayout L = noalloc_layout(tiles, hp->plan.nseg, hp->items.size());
    if (L.total > NOALLOC_SCRATCH_BYTES) {
        f->err = "bakron_solve_noalloc: workspace and work list exceed the 136 MiB static scratch";
        return BAKRON_EINVAL;
    }
    int* ints = reinterpret_cast<int*>(base + L.ints_off);
    int* st_words = reinterpret_cast<int*>(base);
    bk::Workspace ws{reinterpret_cast<float*>(base + L.x_off),
                     reinterpret_cast<float*>(base + L.x_off + L.fbytes), ints, ints + tiles,
                     st_words, st_words + 1};
    // the give-up word is sticky (cleared only by bakron_solve_check); it is
    // cleared once when the device's array is first used, with a fill kernel
    // (no memset node, so a caller may capture this call)
    e = hipSuccess;
    if (first_on_device) e = bk::fill_words(stream, st_words, 2, 0u);
    const int4* items = reinterpret_cast<const int4*>(base + L.items_off);
    if (e == hipSuccess && !hp->items.empty())
        e = hipMemcpyAsync(base + L.items_off, hp->items.data(), sizeof(int4) * hp->items.size(),
                           hipMemcpyHostToDevice, stream);
    int spin_limit = bk::SPIN_LIMIT;
    if (const char* sl = std::getenv("BAKRON_SPIN_LIMIT")) {
        const int v = std::atoi(sl);
        if (v >= 1 && v <= bk::SPIN_LIMIT) spin_limit = v;
    }
    if (e == hipSuccess)
        e = bk::run_plan(stream, nullptr, hp->plan, W, m, n, mt, nt, ws, f->LA, f->LB, f->b_ident,
                         quant_args(q, n), codes, V, nullptr, f->knear, spin_limit, items, nullptr,
                         nullptr, nullptr);
    if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve_noalloc: launch");
    f->noalloc_used = 1;
    f->noalloc_status = st_words;
    return BAKRON_OK;
}

extern "C" bakron_status bakron_solve_check(const bakron_factors* f, hipStream_t stream,
                                           int32_t* failed) {
    if (!f || !failed) return BAKRON_EINVAL;
    bakron_factors* fm = const_cast<bakron_factors*>(f);
    *failed = 0;
    // the handle's own workspace, and the device's static scratch if an
    // allocation-free solve on this handle used it
    int* words[2] = {f->ws_mem ? f->ws.status : nullptr, f->noalloc_used ? f->noalloc_status : nullptr};
    int32_t any = 0;
    for (int* w : words) {
        if (!w) continue;
        int32_t v = 0;
        hipError_t e = hipMemcpyAsync(&v, w, sizeof(v), hipMemcpyDeviceToHost, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        // the status is sticky: clear it once it has been reported
        if (e == hipSuccess && v != 0) {
            e = hipMemsetAsync(w, 0, sizeof(int32_t), stream);
            if (e == hipSuccess) e = hipStreamSynchronize(stream);
        }
        if (e != hipSuccess) return hip_fail(&fm->err, e, "bakron_solve_check");
        any |= v != 0;
    }
    *failed = any;
    return BAKRON_OK;
}
