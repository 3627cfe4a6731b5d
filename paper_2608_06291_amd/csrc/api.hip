// C ABI of libbakron.so: factor handles, the divide-and-conquer schedule and
// the solve driver.  See include/bakron.h for the contract.
#include "common.h"
#include "bakron.h"

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <new>
#include <string>
#include <vector>

namespace bk {
hipError_t factor_one(hipStream_t s, const float* X, int64_t d, double lam, double* Z, double* Ninv,
                      double* T, double* mean, int* fail, int64_t* fail_pivot, float* packed,
                      int64_t nt);
hipError_t pack_identity(hipStream_t s, int64_t nt, float* packed);
hipError_t unpack_factor(hipStream_t s, const float* packed, int64_t d, float* dst);

hipError_t run_schedule(hipStream_t s, const std::vector<SolveOp>& ops, const float* W, int64_t m,
                        int64_t n, int mt, int nt, float* X, float* Y, const float* LA,
                        const float* LB, int b_ident, const float* scale, float qmax,
                        int8_t* codes, float* V, float* pre, int knear, const int4* items,
                        hipEvent_t* evs);
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
    float* X = nullptr;
    float* Y = nullptr;
    int knear = 8;
    std::vector<bk::SolveOp> sched;
    std::vector<int4> items_host;   // node work lists of the schedule
    int4* items = nullptr;
    double prep_bytes = 0.0;
    // measurement hook
    int prof = 0;
    int prof_valid = 0;
    std::vector<hipEvent_t> evs;
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
static double node_alg_flops(const bk::SolveOp& op, int mt, int nt, int knear, int b_ident) {
    double f = 0.0;
    for (int D = op.Mid; D < op.L; ++D) {
        for (int I = imax(0, D - (nt - 1)); I <= imin(D, mt - 1); ++I) {
            const int J = D - I;
            if (!b_ident) f += imax(0, imin(op.Mid - J, I - knear) - imax(op.K - J, 0));
            f += imax(0, imin(op.Mid - I, J - knear) - imax(op.K - I, 0));
        }
    }
    return f * 2.0 * bk::TS * bk::TS * bk::TS;
}

// Work list of one node for MT x MT macro tiles: every (macro tile, push
// kind) with at least one target tile in [Mid, L) and a non-empty source
// range, longest source range first.
static void node_items(int K, int Mid, int L, int mt, int nt, int knear, int b_ident, int MT,
                       std::vector<int4>& out) {
    out.clear();
    const int nmi = (mt + MT - 1) / MT, nmj = (nt + MT - 1) / MT;
    for (int mi = 0; mi < nmi; ++mi) {
        const int I0 = mi * MT;
        // macro columns whose tile anti-diagonals can meet [Mid, L)
        const int mj_lo = imax(0, (Mid - 2 * (MT - 1) - I0 + MT - 1) / MT - 1);
        for (int mj = mj_lo; mj < nmj; ++mj) {
            const int J0 = mj * MT;
            if (I0 + J0 >= L) break;
            bool target = false;
            for (int a = 0; a < MT && !target; ++a)
                for (int b = 0; b < MT && !target; ++b) {
                    const int I = I0 + a, J = J0 + b;
                    target = I < mt && J < nt && I + J >= Mid && I + J < L;
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

static void build_schedule(int K, int L, int mt, int nt, int knear, int b_ident,
                           std::vector<bk::SolveOp>& ops, std::vector<int4>& items) {
    if (L - K == 1) {
        bk::SolveOp op{};
        op.kind = 0;
        op.D = K;
        op.I_lo = K - (nt - 1) > 0 ? K - (nt - 1) : 0;
        const int I_hi = K < mt - 1 ? K : mt - 1;
        op.ntiles = I_hi - op.I_lo + 1;
        // in-tile pairs: sum over entries of (row + column) predecessors
        const double T = bk::TS;
        const double intile = 2.0 * T * T * (T - 1.0);
        double pushes = 0.0;
        for (int I = op.I_lo; I <= I_hi; ++I) {
            const int J = K - I;
            for (int k = 1; k <= knear; ++k) {
                if (!b_ident && I + k < mt) pushes += 1.0;
                if (J + k < nt) pushes += 1.0;
            }
        }
        op.flops = op.ntiles * intile + pushes * 2.0 * T * T * T;
        op.mfma_flops = pushes * 2.0 * T * T * T;
        ops.push_back(op);
        return;
    }
    const int Mid = (K + L) / 2;
    build_schedule(K, Mid, mt, nt, knear, b_ident, ops, items);
    if (L - K > knear + 1) {
        bk::SolveOp op{};
        op.kind = 1;
        op.K = K;
        op.Mid = Mid;
        op.L = L;
        std::vector<int4> its;
        // 128 x 128 workgroups when they fill the chip twice over, else 64 x 64
        op.macro = bk::MACRO;
        node_items(K, Mid, L, mt, nt, knear, b_ident, 4, its);
        if ((int)its.size() < 512) {
            op.macro = 2;
            node_items(K, Mid, L, mt, nt, knear, b_ident, 2, its);
        }
        if (!its.empty()) {
            op.item_off = (int)items.size();
            op.item_cnt = (int)its.size();
            const double chunk = 2.0 * (op.macro * bk::TS) * (op.macro * bk::TS) * bk::TS;
            op.mfma_flops = 0.0;
            for (const int4& it : its) op.mfma_flops += (it.w - (it.z >> 1)) * chunk;
            op.flops = node_alg_flops(op, mt, nt, knear, b_ident);
            items.insert(items.end(), its.begin(), its.end());
            ops.push_back(op);
        }
    }
    build_schedule(Mid, L, mt, nt, knear, b_ident, ops, items);
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
    if (const char* kn = std::getenv("BAKRON_KNEAR")) {
        int v = std::atoi(kn);
        if (v >= 0 && v <= 8) f->knear = v;
    }

    const int64_t dmax = (B && m > n) ? m : n;
    const int64_t ntA = cdiv(n, bk::TS);
    double *Z = nullptr, *Ninv = nullptr, *T = nullptr, *scal = nullptr;
    int* flags = nullptr;
    bakron_status st = BAKRON_OK;
    hipError_t e;
    auto cleanup = [&]() {
        if (Z) hipFree(Z);
        if (Ninv) hipFree(Ninv);
        if (T) hipFree(T);
        if (scal) hipFree(scal);
        if (flags) hipFree(flags);
    };
    const size_t zbytes = sizeof(double) * (size_t)dmax * (size_t)dmax;
    const size_t tbytes = sizeof(double) * ((size_t)dmax * (size_t)dmax / 4 + (size_t)dmax * 64 +
                                            64 * 64 + 64);
    if ((e = hipMalloc(&Z, zbytes)) != hipSuccess || (e = hipMalloc(&Ninv, zbytes)) != hipSuccess ||
        (e = hipMalloc(&T, tbytes)) != hipSuccess ||
        (e = hipMalloc(&scal, 4 * sizeof(double))) != hipSuccess ||
        (e = hipMalloc(&flags, 8 * sizeof(int64_t))) != hipSuccess) {
        st = hip_fail(&g_last_error, e, "bakron_factor: hipMalloc (factor scratch)");
        cleanup();
        delete f;
        return st;
    }
    e = hipMemsetAsync(flags, 0, 8 * sizeof(int64_t), stream);
    if (e == hipSuccess)
        e = hipMalloc(&f->LA, sizeof(float) * (size_t)(ntA * (ntA + 1) / 2) * bk::TILE_ELEMS);
    if (e == hipSuccess)
        e = bk::factor_one(stream, A, n, (double)damp, Z, Ninv, T, scal, flags,
                           reinterpret_cast<int64_t*>(flags) + 2, f->LA, ntA);
    if (e == hipSuccess && B) {
        const int64_t mtB = cdiv(m, bk::TS);
        f->LB_tiles = mtB;
        e = hipMalloc(&f->LB, sizeof(float) * (size_t)(mtB * (mtB + 1) / 2) * bk::TILE_ELEMS);
        if (e == hipSuccess)
            e = bk::factor_one(stream, B, m, (double)damp, Z, Ninv, T, scal + 1, flags + 1,
                               reinterpret_cast<int64_t*>(flags) + 3, f->LB, mtB);
    }
    if (e != hipSuccess) {
        st = hip_fail(&g_last_error, e, "bakron_factor: launch");
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
    if (f->X) hipFree(f->X);
    if (f->Y) hipFree(f->Y);
    if (f->items) hipFree(f->items);
    for (hipEvent_t ev : f->evs) hipEventDestroy(ev);
    if (cur != f->device) hipSetDevice(cur);
    delete f;
}

static bakron_status ensure_workspace(bakron_factors* f, int64_t m, int64_t n) {
    if (f->ws_m == m && f->ws_n == n && f->X) return BAKRON_OK;
    const int64_t mt = cdiv(m, bk::TS), nt = cdiv(n, bk::TS);
    if (f->X) { hipFree(f->X); f->X = nullptr; }
    if (f->Y) { hipFree(f->Y); f->Y = nullptr; }
    f->ws_m = f->ws_n = -1;
    const size_t bytes = sizeof(float) * (size_t)mt * (size_t)nt * bk::TILE_ELEMS;
    hipError_t e = hipMalloc(&f->X, bytes);
    if (e == hipSuccess) e = hipMalloc(&f->Y, bytes);
    if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: hipMalloc (workspace)");
    // identity B grows to the requested m
    if (f->b_ident && f->LB_tiles < mt) {
        if (f->LB) hipFree(f->LB);
        f->LB = nullptr;
        e = hipMalloc(&f->LB, sizeof(float) * (size_t)(mt * (mt + 1) / 2) * bk::TILE_ELEMS);
        if (e == hipSuccess) e = bk::pack_identity(0, mt, f->LB);
        if (e == hipSuccess) e = hipDeviceSynchronize();
        if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: identity factor");
        f->LB_tiles = mt;
    }
    f->sched.clear();
    f->items_host.clear();
    build_schedule(0, (int)(mt + nt - 1), (int)mt, (int)nt, f->knear, f->b_ident, f->sched,
                   f->items_host);
    if (f->items) { hipFree(f->items); f->items = nullptr; }
    if (!f->items_host.empty()) {
        const size_t ib = sizeof(int4) * f->items_host.size();
        e = hipMalloc(&f->items, ib);
        if (e == hipSuccess) e = hipMemcpy(f->items, f->items_host.data(), ib, hipMemcpyHostToDevice);
        if (e != hipSuccess) return hip_fail(&f->err, e, "bakron_solve: work list upload");
    }
    f->prep_bytes = (double)m * n * 4.0 + 2.0 * 4.0 * mt * nt * bk::TILE_ELEMS;
    f->ws_m = m;
    f->ws_n = n;
    return BAKRON_OK;
}

static bakron_status solve_impl(const float* W, int64_t m, int64_t n, const bakron_factors* fc,
                                bakron_quantizer q, int8_t* codes, float* V, float* pre,
                                hipStream_t stream) {
    bakron_factors* f = const_cast<bakron_factors*>(fc);
    if (!f) return BAKRON_EINVAL;
    f->err.clear();
    if (!W || !codes || !V || !q.scale || m <= 0 || n <= 0) {
        f->err = "bakron_solve: null pointer or non-positive size";
        return BAKRON_EINVAL;
    }
    if (n != f->n || (!f->b_ident && m != f->m)) {
        f->err = "bakron_solve: (m, n) does not match the factor handle";
        return BAKRON_EINVAL;
    }
    if (q.bits < 2 || q.bits > 8) {
        f->err = "bakron_solve: bits must be in [2, 8]";
        return BAKRON_EINVAL;
    }
    if ((m + bk::TS) * (n + bk::TS) > ((int64_t)1 << 40)) {
        f->err = "bakron_solve: matrix too large";
        return BAKRON_EINVAL;
    }
    bakron_status st = ensure_workspace(f, m, n);
    if (st != BAKRON_OK) return st;
    const int mt = (int)cdiv(m, bk::TS), nt = (int)cdiv(n, bk::TS);
    const float qmax = (float)((1 << (q.bits - 1)) - 1);
    hipEvent_t* evs = nullptr;
    f->prof_valid = 0;
    if (f->prof) {
        const size_t need = 2 * (f->sched.size() + 1);
        while (f->evs.size() < need) {
            hipEvent_t ev;
            hipError_t ee = hipEventCreate(&ev);
            if (ee != hipSuccess) return hip_fail(&f->err, ee, "bakron_solve: hipEventCreate");
            f->evs.push_back(ev);
        }
        evs = f->evs.data();
    }
    hipError_t e = bk::run_schedule(stream, f->sched, W, m, n, mt, nt, f->X, f->Y, f->LA, f->LB,
                                    f->b_ident, q.scale, qmax, codes, V, pre, f->knear, f->items,
                                    evs);
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

extern "C" bakron_status bakron_profile_read(const bakron_factors* f, bakron_kernel_stat* prep,
                                            bakron_kernel_stat* leaf, bakron_kernel_stat* node) {
    if (!f || !prep || !leaf || !node) return BAKRON_EINVAL;
    if (!f->prof_valid) return BAKRON_EINVAL;
    bakron_kernel_stat* outs[3] = {prep, leaf, node};
    for (bakron_kernel_stat* o : outs) *o = bakron_kernel_stat{0.0, 0, 0.0, 0.0};
    float ms = 0.0f;
    hipError_t e = hipEventElapsedTime(&ms, f->evs[0], f->evs[1]);
    if (e != hipSuccess) return hip_fail(&const_cast<bakron_factors*>(f)->err, e, "bakron_profile_read");
    prep->ms = ms;
    prep->launches = 1;
    prep->flops = f->prep_bytes;  // bytes moved (the prep kernel does no arithmetic)
    for (size_t i = 0; i < f->sched.size(); ++i) {
        e = hipEventElapsedTime(&ms, f->evs[2 * (i + 1)], f->evs[2 * (i + 1) + 1]);
        if (e != hipSuccess)
            return hip_fail(&const_cast<bakron_factors*>(f)->err, e, "bakron_profile_read");
        bakron_kernel_stat* o = f->sched[i].kind == 0 ? leaf : node;
        o->ms += ms;
        o->launches += 1;
        o->flops += f->sched[i].flops;
        o->mfma_flops += f->sched[i].mfma_flops;
    }
    return BAKRON_OK;
}
