// host.cpp -- the C ABI declared in include/lapattn.h: argument validation, workspace
// planning, launch sequencing on the caller's stream, optional per-kernel timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <initializer_list>
#include <mutex>
#include <new>
#include <vector>

#include "lapattn.h"
#include "kernels.hpp"

namespace {

constexpr int kMaxM = 128;
constexpr int kMaxT = 64;
constexpr int kKeyChunk = 256;   // keys per block of the fp32 key-summary kernel (one 64-key tile per wave) ...
constexpr int kKeyMaxChunk = 1024;  // ... up to this many for long sequences (a multiple of 256)
constexpr int kLmChunk = 256;    // tokens per block of the landmark-major backward passes (at most)
constexpr int kLmMinChunk = 32;  // ... and at least
constexpr int kMaxParts = 64;    // partial sums per head that a shorter chunk may create
constexpr int kLmWaves = 1024;   // one wave per SIMD of the chip
constexpr int kDwcChunk = 256;   // tokens per block of the convolution filter gradient
constexpr int kDwcMaxK = 7;      // largest convolution filter side

// ------------------------------------------------------------------------------- validation

int check_shape(int B, int H, int n, int d, int m, float lambda, int T, int dtype, int norm, float eps) {
    if (B < 1 || H < 1 || n < 1 || m < 1 || m > n) return LAPATTN_ERR_SHAPE;
    if ((long long)B * H * (long long)n * (d > 0 ? d : 1) >= (1LL << 31)) return LAPATTN_ERR_SHAPE;
    if (!(std::isfinite(lambda) && lambda > 0.f)) return LAPATTN_ERR_PARAM;
    if (T < 0 || T > kMaxT) return LAPATTN_ERR_PARAM;
    if (dtype != LAPATTN_FP32 && dtype != LAPATTN_BF16) return LAPATTN_ERR_PARAM;
    if (norm != LAPATTN_NORM_INLINE && norm != LAPATTN_NORM_ROWSUM && norm != LAPATTN_NORM_NONE &&
        norm != LAPATTN_NORM_MSPACE)
        return LAPATTN_ERR_PARAM;
    if (!(std::isfinite(eps) && eps >= 0.f)) return LAPATTN_ERR_PARAM;
    if (d != 32 && d != 64) return LAPATTN_ERR_UNSUPPORTED;
    if (m > kMaxM) return LAPATTN_ERR_UNSUPPORTED;
    return LAPATTN_OK;
}

// Tensors are read and written in 16-byte vectors; workspace slices are carved at 256-byte offsets.
bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int check_align(std::initializer_list<const void*> tensors, const void* workspace) {
    for (const void* t : tensors)
        if (!aligned(t, 16)) return LAPATTN_ERR_ALIGN;
    if (workspace && !aligned(workspace, 256)) return LAPATTN_ERR_ALIGN;
    return LAPATTN_OK;
}

// ------------------------------------------------------------------------------- workspace plan

struct FastPlan {
    size_t qt, kt, vseg, segmax, vsegmax, frame, qfix, kfix, kcen, vbar, XT, cinfo, Upart, Mt, mscale, Mones, M;
    size_t vpart;  // split key side: value sums per key block [BH][nkb][d]
    size_t E;      // convolution branch: DWC(V) + bias, fp32 [BH][n][d]
    size_t mvec;   // landmark-space normalisation: [BH][2][d]
    size_t total;
    int kpb, nkb;
    bool split;    // key side with the landmarks split over the waves (key2_kernel), T tiles per head
    int T;
};

struct Plan {
    size_t qt, kt, Upart, vpart, Xs, cinfo, U, M, Mc, vbar;              // forward
    size_t Ebuf, Ud, nsbs, dDW;          // m > 64: solve and its backward spread over workgroups
    size_t pool_part;                    // landmark sums split over blocks (small m BH)
    size_t oF;                           // bf16 forward with m > 64: the fp32 output
    size_t Aq, dDq, rs, dYd, dvbar_part, dM_part, dkt_part, dU, dvbar,   // backward
        dqtW, dkpool, dDk, dqt_part;
    size_t wQ, wK, wV, wG, gQ, gK, gV;   // bf16 backward: fp32 copies of the inputs, fp32 gradients
    size_t E;                            // convolution branch, forward: DWC(V) + bias [BH][n][d]
    size_t mvec;                         // landmark-space normalisation: [BH][2][d]
    size_t p0_part;                      // landmark-space normalisation: per-block sums of dOut
    size_t dwc_part;                     // convolution branch, backward: filter-gradient partials
    size_t total;
    int MP, ng, nkc, nqb, nlc, lmc, kc;
};

// Keys per block of the fp32 key-side summary: 256 (many small blocks fill the three block slots
// of every compute unit evenly), doubled while a head would have more than kMaxParts partial sums.
int key_chunk(int n) {
    int c = kKeyChunk;
    while (c < kKeyMaxChunk && (n + c - 1) / c > kMaxParts) c *= 2;
    return c;
}

// Tokens per block of the landmark-major backward passes (one wave each, walking its tokens in
// order): 256, halved while the grid holds fewer waves than the chip has SIMDs and the number of
// per-head partial sums stays within kMaxParts, so that a few heads still spread over the chip.
int lm_chunk(int BH, int n) {
    int c = kLmChunk;
    while (c > kLmMinChunk && (long long)BH * ((n + c - 1) / c) < kLmWaves &&
           (n + c / 2 - 1) / (c / 2) <= kMaxParts)
        c /= 2;
    return c;
}

struct Carver {
    size_t off = 0;
    size_t take(size_t bytes) {
        off = (off + 255) & ~size_t(255);
        size_t o = off;
        off += bytes;
        return o;
    }
};

Plan make_plan(int BH, int n, int d, int m, int T, bool bwd, bool bf16 = false, bool dwc = false) {
    Plan p{};
    p.MP = m <= 32 ? 32 : (m <= 64 ? 64 : 128);
    p.ng = (m + 63) / 64;   // landmark groups of 64 (the row arrays below are group-major)
    const bool big = p.MP == 128;
    p.kc = key_chunk(n);
    p.nkc = (n + p.kc - 1) / p.kc;
    p.nqb = (n + 255) / 256;
    p.lmc = lm_chunk(BH, n);
    p.nlc = (n + p.lmc - 1) / p.lmc;
    const size_t bh = (size_t)BH, d1 = (size_t)d + 1, f = sizeof(float), g = sizeof(double);
    const size_t mpp = (size_t)p.MP * p.MP;
    Carver c;
    p.qt = c.take(bh * m * d * f);
    p.kt = c.take(bh * m * d * f);
    p.pool_part = c.take(bh * m * (size_t)lapattn::pool_split(BH, n, m) * 2 * d * g);
    p.Upart = c.take(bh * p.nkc * m * d1 * f);
    p.vpart = c.take(bh * p.nkc * (size_t)d * f);
    // X_0..X_T and W for the backward (always, for m > 64)
    p.Xs = c.take(bh * ((bwd || big) ? (size_t)T + 2 : 1) * mpp * g);
    p.cinfo = c.take(bh * 4 * g);
    p.U = c.take(bh * m * d1 * f);
    p.M = c.take(bh * m * d1 * f);
    p.Mc = c.take(bh * m * d * f);
    p.vbar = c.take(bh * d * f);
    p.mvec = c.take(bh * 2 * d * f);
    if (big) {
        p.Ebuf = c.take(bh * 2 * mpp * g);
        p.Ud = c.take(bh * m * d1 * g);
    }
    const size_t rows = bh * p.ng * n * 64 * f;   // [BH][ng][n][64]: rows of pitch 64 (16-byte aligned)
    if (bwd) {
        p.Aq = c.take(rows);
        p.dDq = c.take(rows);
        p.rs = c.take(bh * n * f);
        p.dYd = c.take(bh * n * f);
        p.dvbar_part = c.take(bh * p.nqb * d * f);
        p.p0_part = c.take(bh * p.nqb * d * f);
        p.dM_part = c.take(bh * p.nlc * m * d1 * f);
        p.dkt_part = c.take(bh * p.nlc * m * d * f);
        p.dU = c.take(bh * m * d1 * f);
        p.dvbar = c.take(bh * d * f);
        p.dqtW = c.take(bh * m * d * f);
        p.dkpool = c.take(bh * m * d * f);
        p.dDk = c.take(rows);
        if (big) p.nsbs = c.take(lapattn::nsb_backward_scratch(BH, d) * g);
        p.dDW = c.take(bh * mpp * f);
        p.dqt_part = c.take(bh * p.nlc * m * d * f);
        if (bf16) {
            const size_t t = bh * n * d * f;
            p.wQ = c.take(t);
            p.wK = c.take(t);
            p.wV = c.take(t);
            p.wG = c.take(t);
            p.gQ = c.take(t);
            p.gK = c.take(t);
            p.gV = c.take(t);
        }
        if (dwc)
            p.dwc_part = c.take(bh * ((n + kDwcChunk - 1) / kDwcChunk) * d * (kDwcMaxK * kDwcMaxK + 1) * f);
    }
    if (bf16 && !bwd) {   // the bf16 forward with m > 64: fp32 copies of the inputs, fp32 output
        const size_t t = bh * n * d * f;
        p.wQ = c.take(t);
        p.wK = c.take(t);
        p.wV = c.take(t);
        p.oF = c.take(t);
    }
    if (dwc) p.E = c.take(bh * n * d * f);
    p.total = (c.off + 255) & ~size_t(255);
    return p;
}

// The bf16 forward: key blocks of kpb keys (a multiple of 256), sized so the key-side launch
// has about two 64-key tiles per wave when the work allows it.
FastPlan make_fast_plan(int BH, int n, int d, int m, bool dwc = false) {
    FastPlan p{};
    p.split = m > 48;
    if (p.split) {
        // chunks per head: the fewest (rounds of blocks over the chip's block slots) x (tiles per
        // block), three blocks per CU at d = 64, four at d = 32, less the BH slots of the blocks
        // that solve Newton-Schulz in the same launch; on a tie the fewest rounds, then the most
        // blocks
        p.T = (n + 127) / 128;
        const long long slots = std::max(256LL, 256LL * (d == 32 ? 4 : 3) - BH);
        long long best = -1, best_rounds = 0;
        for (int c = 1; c <= p.T; ++c) {
            const long long rounds = ((long long)BH * c + slots - 1) / slots;
            const long long cost = rounds * ((p.T + c - 1) / c);
            if (best < 0 || cost < best || (cost == best && rounds <= best_rounds)) {
                best = cost;
                best_rounds = rounds;
                p.nkb = c;
            }
        }
        p.kpb = 0;
    } else {
        const long long tiles = (long long)BH * ((n + 63) / 64);
        const long long per_wave = tiles / 2048 > 1 ? tiles / 2048 : 1;
        p.kpb = (int)(256 * per_wave);
        p.nkb = (n + p.kpb - 1) / p.kpb;
    }
    const size_t bh = (size_t)BH, d1 = (size_t)d + 1, f = sizeof(float), g = sizeof(double);
    Carver c;
    p.qt = c.take(bh * m * d * f);
    p.kt = c.take(bh * m * d * f);
    p.vseg = c.take(bh * m * d * g);
    p.segmax = c.take(bh * m * f);
    p.vsegmax = c.take(bh * m * f);
    p.frame = c.take(bh * 8 * f);
    p.qfix = c.take(bh * 64 * (d / 2) * 4);
    p.kfix = c.take(bh * 64 * (d / 2) * 4);
    p.kcen = c.take(bh * (d / 2) * 4);
    p.vbar = c.take(bh * d * f);
    p.XT = c.take(bh * 64 * 64 * f);
    p.cinfo = c.take(bh * 4 * f);
    p.Upart = c.take(bh * p.nkb * d1 * 64 * f);   // [h][kb][c][a], 64 rows a
    p.vpart = c.take(bh * p.nkb * (size_t)d * f);
    p.Mt = c.take(bh * 4 * ((size_t)d / 32) * 512 * 2);
    p.mscale = c.take(bh * ((size_t)d / 8 + 1) * f);
    p.Mones = c.take(bh * 64 * f);
    p.M = c.take(bh * m * d1 * f);
    p.mvec = c.take(bh * 2 * d * f);
    if (dwc) p.E = c.take(bh * n * d * f);
    p.total = (c.off + 255) & ~size_t(255);
    return p;
}

template <typename T>
T* at(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// ------------------------------------------------------------------------------- timing

struct Timing {
    std::mutex mu;
    bool enabled = false;
    std::vector<const char*> names;
    std::vector<hipEvent_t> ev;   // 2 per kernel of the last call
    size_t used = 0;
};

Timing& timing() {
    static Timing* t = new Timing();
    return *t;
}

// Records one (start, stop) pair around each launch while timing is enabled; the
// record accumulates over calls until timing is enabled again.
class Recorder {
  public:
    explicit Recorder(hipStream_t st) : st_(st) {
        Timing& t = timing();
        std::lock_guard<std::mutex> g(t.mu);
        on_ = t.enabled;
    }
    hipError_t run(const char* name, hipError_t (*fn)(void*), void* ctx) {
        if (!on_) return fn(ctx);
        Timing& t = timing();
        std::lock_guard<std::mutex> g(t.mu);
        while (t.ev.size() < t.used + 2) {
            hipEvent_t e;
            hipError_t err = hipEventCreate(&e);
            if (err != hipSuccess) return err;
            t.ev.push_back(e);
        }
        hipEvent_t a = t.ev[t.used], b = t.ev[t.used + 1];
        hipError_t err = hipEventRecord(a, st_);
        if (err != hipSuccess) return err;
        err = fn(ctx);
        if (err != hipSuccess) return err;
        err = hipEventRecord(b, st_);
        t.used += 2;
        t.names.push_back(name);
        return err;
    }

  private:
    hipStream_t st_;
    bool on_ = false;
};

// A launch is a lambda captured by reference; this adapter turns it into (fn, ctx).
template <typename F>
hipError_t run_named(Recorder& rec, const char* name, F&& f) {
    return rec.run(name, [](void* ctx) -> hipError_t { return (*static_cast<F*>(ctx))(); }, (void*)&f);
}

int norm_of(const lapattn_opts* o) { return o ? o->norm : LAPATTN_NORM_INLINE; }
float eps_of(const lapattn_opts* o) { return o ? o->eps : 0.f; }
const float* whiten_of(const lapattn_opts* o) { return o ? o->whiten : nullptr; }
bool save_of(const lapattn_opts* o) { return o && o->save; }
lapattn::LmPool pool_of(const lapattn_opts* o) { return o ? lapattn::LmPool{o->grid_w, o->pool_r} : lapattn::LmPool{0, 0}; }

// Token map and landmark geometry: no map (gw = 0) or a row-major map of width gw dividing n;
// segments (r = 0), or r x r windows of the map, r dividing both sides, with
// m = (n / gw / r)(gw / r) windows.
int check_pool(int n, int m, lapattn::LmPool pl) {
    if (pl.gw < 0 || pl.r < 0 || (pl.r > 0 && pl.gw == 0)) return LAPATTN_ERR_PARAM;
    if (pl.gw > 0 && n % pl.gw) return LAPATTN_ERR_SHAPE;
    if (pl.r == 0) return LAPATTN_OK;
    if ((n / pl.gw) % pl.r || pl.gw % pl.r) return LAPATTN_ERR_SHAPE;
    if ((long long)m != (long long)(n / pl.gw / pl.r) * (pl.gw / pl.r)) return LAPATTN_ERR_SHAPE;
    return LAPATTN_OK;
}

// The convolution branch of Eq. (7).
struct Dwc {
    int k;
    const float *w, *b;
    float *dw, *db;
};
Dwc dwc_of(const lapattn_opts* o) {
    return o ? Dwc{o->dwc_k, o->dwc_w, o->dwc_b, o->dwc_dw, o->dwc_db} : Dwc{0, nullptr, nullptr, nullptr, nullptr};
}
int check_dwc(const Dwc& c, lapattn::LmPool pl) {
    if (c.k == 0) return LAPATTN_OK;
    if (c.k < 0 || c.k > kDwcMaxK || c.k % 2 == 0 || pl.gw < 1) return LAPATTN_ERR_PARAM;
    if (!c.w) return LAPATTN_ERR_NULL;
    return LAPATTN_OK;
}

// The forward stages shared by lapattn_forward and lapattn_backward (which recomputes them).
hipError_t forward_internals(Recorder& rec, const Plan& p, const void* Q, const void* K, const void* V, void* ws,
                             int BH, int n, int d, int m, float lambda, int T, int dtype, float eps, bool store_all,
                             lapattn::LmPool pl, hipStream_t st, float* Bsave = nullptr) {
    float* qt = at<float>(ws, p.qt);
    float* kt = at<float>(ws, p.kt);
    float* Upart = at<float>(ws, p.Upart);
    float* vpart = at<float>(ws, p.vpart);
    hipError_t e;
    e = run_named(rec, "pool", [&] {
        return lapattn::launch_pool(dtype, Q, K, qt, kt, at<double>(ws, p.pool_part), BH, n, d, m, pl, st);
    });
    if (e != hipSuccess) return e;
    e = run_named(rec, "key_summary", [&] {
        return lapattn::launch_key_summary(dtype, K, V, qt, Upart, vpart, Bsave, BH, n, d, m, lambda, p.kc, p.nkc,
                                           st);
    });
    if (e != hipSuccess) return e;
    if (p.MP == 128)
        return run_named(rec, "ns_solve", [&] {
            return lapattn::launch_nsb_forward(qt, kt, Upart, vpart, at<double>(ws, p.Xs), at<double>(ws, p.Ebuf),
                                               at<double>(ws, p.Ud), at<double>(ws, p.cinfo), at<float>(ws, p.U),
                                               at<float>(ws, p.M), at<float>(ws, p.Mc), at<float>(ws, p.vbar), BH, n,
                                               d, m, T, (double)lambda, (double)eps, p.nkc, st);
        });
    e = run_named(rec, "ns_solve", [&] {
        return lapattn::launch_ns_solve(qt, kt, Upart, vpart, at<double>(ws, p.Xs), at<double>(ws, p.cinfo),
                                        at<float>(ws, p.U), at<float>(ws, p.M), at<float>(ws, p.Mc),
                                        at<float>(ws, p.vbar), BH, n, d, m, T,
                                        (double)lambda, (double)eps, p.nkc, store_all ? 1 : 0, p.MP, st);
    });
    return e;
}

hipError_t forward_fast(Recorder& rec, const FastPlan& p, const void* Q, const void* K, const void* V, void* Out,
                        void* ws, int BH, int H, int n, int d, int m, float lambda, int T, int norm, float eps,
                        lapattn::LmPool pl, const Dwc& dwc, const float* whiten, hipStream_t st) {
    const bool mspace = norm == LAPATTN_NORM_MSPACE;
    hipError_t e;
    // the convolution branch: 3 x 3 filters are formed in the query kernel's epilogue; other
    // sizes by the separate stencil kernel into E, which the query kernel adds
    const bool dwc_fused = dwc.k == 3;
    float* E = (dwc.k && !dwc_fused) ? at<float>(ws, p.E) : nullptr;
    if (E) {
        e = run_named(rec, "dwc", [&] {
            return lapattn::launch_dwc_fwd(lapattn::DT_BF16, V, dwc.w, dwc.b, E, BH, H, n, d, pl.gw, dwc.k, st);
        });
        if (e != hipSuccess) return e;
    }
    e = run_named(rec, "pool", [&] {
        return lapattn::launch_fast_pool(Q, K, V, at<float>(ws, p.qt), at<float>(ws, p.kt), at<double>(ws, p.vseg),
                                         at<float>(ws, p.segmax), at<float>(ws, p.vsegmax), BH, n, d, m, pl, st);
    });
    if (e != hipSuccess) return e;
    e = run_named(rec, "frame_ns", [&] {
        return lapattn::launch_fast_frame_ns(at<float>(ws, p.qt), at<float>(ws, p.kt), at<double>(ws, p.vseg),
                                             at<float>(ws, p.segmax), at<float>(ws, p.vsegmax), at<float>(ws, p.frame),
                                             at<uint32_t>(ws, p.qfix), at<uint32_t>(ws, p.kfix), at<float>(ws, p.vbar),
                                             at<float>(ws, p.XT), at<float>(ws, p.cinfo), BH, n, d, m, lambda, T, eps,
                                             st);
    });
    if (e != hipSuccess) return e;
    e = run_named(rec, "key", [&] {
        if (p.split)
            return lapattn::launch_fast_key2(K, V, at<uint32_t>(ws, p.qfix), at<uint32_t>(ws, p.kfix),
                                             at<float>(ws, p.frame), at<float>(ws, p.Upart), at<float>(ws, p.vpart),
                                             at<float>(ws, p.XT),
                                             at<float>(ws, p.cinfo), at<uint32_t>(ws, p.kcen), BH, n, d, m, p.T,
                                             p.nkb, T, eps, st);
        return lapattn::launch_fast_key(K, V, at<uint32_t>(ws, p.qfix), at<float>(ws, p.frame), at<float>(ws, p.Upart),
                                        BH, n, d, m, p.kpb, p.nkb, st);
    });
    if (e != hipSuccess) return e;
    e = run_named(rec, "m_final", [&] {
        return lapattn::launch_fast_mfinal(at<float>(ws, p.Upart), at<float>(ws, p.XT), at<_Float16>(ws, p.Mt),
                                           at<float>(ws, p.mscale), at<float>(ws, p.Mones), at<float>(ws, p.M), BH, d, m,
                                           p.nkb, whiten, mspace ? 1 : 0, H, at<float>(ws, p.mvec),
                                           at<float>(ws, p.vbar), p.split ? at<float>(ws, p.vpart) : nullptr, n,
                                           norm == LAPATTN_NORM_INLINE ? 1 : 0,
                                           p.split ? nullptr : at<uint32_t>(ws, p.kfix), at<uint32_t>(ws, p.kcen),
                                           at<float>(ws, p.frame),
                                           st);
    });
    if (e != hipSuccess) return e;
    e = run_named(rec, "query", [&] {
        return lapattn::launch_fast_query(norm, Q, Out, at<uint32_t>(ws, p.kfix), at<uint32_t>(ws, p.kcen),
                                          at<float>(ws, p.frame), at<_Float16>(ws, p.Mt), at<float>(ws, p.mscale),
                                          at<float>(ws, p.Mones), at<float>(ws, p.vbar), E, at<float>(ws, p.mvec), BH,
                                          n, d, m, V, dwc_fused ? dwc.w : nullptr, dwc_fused ? dwc.b : nullptr, pl.gw,
                                          H, st);
    });
    return e;
}

}  // namespace

extern "C" {

size_t lapattn_workspace_size(int B, int H, int n, int d, int m, int ns_iters, int dtype, int flags) {
    if (check_shape(B, H, n, d, m, 1.f, ns_iters, dtype, LAPATTN_NORM_INLINE, 0.f) != LAPATTN_OK) return 0;
    if (flags & ~(LAPATTN_WS_BACKWARD | LAPATTN_WS_DWC)) return 0;
    const bool bwd = (flags & LAPATTN_WS_BACKWARD) != 0, dwc = (flags & LAPATTN_WS_DWC) != 0;
    if (dtype == LAPATTN_BF16 && !bwd && m <= 64) return make_fast_plan(B * H, n, d, m, dwc).total;
    return make_plan(B * H, n, d, m, ns_iters, bwd, dtype == LAPATTN_BF16, dwc).total;
}

int lapattn_forward(const void* Q, const void* K, const void* V, void* Out, int B, int H, int n, int d, int m,
                    float lambda, int ns_iters, int dtype, const lapattn_opts* opts, void* workspace,
                    size_t workspace_bytes, lapattn_stream_t stream) {
    try {
        if (!Q || !K || !V || !Out) return LAPATTN_ERR_NULL;
        const int norm = norm_of(opts);
        const float eps = eps_of(opts);
        const lapattn::LmPool pl = pool_of(opts);
        const Dwc dwc = dwc_of(opts);
        int rc = check_shape(B, H, n, d, m, lambda, ns_iters, dtype, norm, eps);
        if (rc) return rc;
        if ((rc = check_pool(n, m, pl))) return rc;
        if ((rc = check_dwc(dwc, pl))) return rc;
        rc = check_align({Q, K, V, Out}, workspace);
        if (rc) return rc;
        const int BH = B * H;
        hipStream_t st = reinterpret_cast<hipStream_t>(stream);
        if (dtype == LAPATTN_BF16 && m <= 64) {
            const FastPlan fp = make_fast_plan(BH, n, d, m, dwc.k != 0);
            if (!workspace || workspace_bytes < fp.total) return LAPATTN_ERR_WORKSPACE;
            Recorder rec(st);
            hipError_t e = forward_fast(rec, fp, Q, K, V, Out, workspace, BH, H, n, d, m, lambda, ns_iters, norm, eps,
                                        pl, dwc, whiten_of(opts), st);
            return e == hipSuccess ? LAPATTN_OK : LAPATTN_ERR_HIP;
        }
        // small heads (fp32): one launch per forward, every intermediate in LDS
        if (dtype == LAPATTN_FP32 && n <= 256 && m <= 32 && (d == 32 || d == 64) && !save_of(opts) && dwc.k == 0 &&
            norm != LAPATTN_NORM_MSPACE) {
            const Plan p = make_plan(BH, n, d, m, ns_iters, false, false, false);
            if (!workspace || workspace_bytes < p.total) return LAPATTN_ERR_WORKSPACE;
            Recorder rec(st);
            const hipError_t e = run_named(rec, "small_forward", [&] {
                return lapattn::launch_small_forward(norm, static_cast<const float*>(Q), static_cast<const float*>(K),
                                                     static_cast<const float*>(V), static_cast<float*>(Out), BH, n, d,
                                                     m, lambda, ns_iters, eps, pl, st);
            });
            return e == hipSuccess ? LAPATTN_OK : LAPATTN_ERR_HIP;
        }
        // bf16 inputs with m > 64: widened to fp32 (exact), the fp32 path, the output rounded to bf16
        const bool bf16 = dtype == LAPATTN_BF16;
        // save: the backward's layout, with every Newton-Schulz iterate kept, so that a following
        // lapattn_backward (save set, same arguments and workspace) can skip the recomputation
        const bool save = !bf16 && save_of(opts);
        const Plan p = make_plan(BH, n, d, m, ns_iters, save, bf16, dwc.k != 0);
        if (!workspace || workspace_bytes < p.total) return LAPATTN_ERR_WORKSPACE;
        Recorder rec(st);
        hipError_t e;
        const void* q = Q;
        const void* k = K;
        const void* v = V;
        void* out = Out;
        if (bf16) {
            e = run_named(rec, "widen", [&] {
                return lapattn::launch_widen_bf16(static_cast<const uint16_t*>(Q), static_cast<const uint16_t*>(K),
                                                  static_cast<const uint16_t*>(V), nullptr, at<float>(workspace, p.wQ),
                                                  at<float>(workspace, p.wK), at<float>(workspace, p.wV), nullptr,
                                                  (size_t)BH * n * d, st);
            });
            if (e != hipSuccess) return LAPATTN_ERR_HIP;
            q = at<float>(workspace, p.wQ);
            k = at<float>(workspace, p.wK);
            v = at<float>(workspace, p.wV);
            out = at<float>(workspace, p.oF);
        }
        // with save the key side also leaves B's rows (in the backward's dDk slice) and the query
        // side A's rows (Aq), so that the backward skips its two distance passes as well
        e = forward_internals(rec, p, q, k, v, workspace, BH, n, d, m, lambda, ns_iters, LAPATTN_FP32, eps, save, pl,
                              st, save ? at<float>(workspace, p.dDk) : nullptr);
        if (e != hipSuccess) return LAPATTN_ERR_HIP;
        float* E = dwc.k ? at<float>(workspace, p.E) : nullptr;
        if (E) {
            e = run_named(rec, "dwc", [&] {
                return lapattn::launch_dwc_fwd(lapattn::DT_F32, v, dwc.w, dwc.b, E, BH, H, n, d, pl.gw, dwc.k, st);
            });
            if (e != hipSuccess) return LAPATTN_ERR_HIP;
        }
        if (norm == LAPATTN_NORM_MSPACE) {
            e = run_named(rec, "mspace_vec", [&] {
                return lapattn::launch_mspace_vec(at<float>(workspace, p.M), whiten_of(opts),
                                                  at<float>(workspace, p.mvec), BH, H, d, m, st);
            });
            if (e != hipSuccess) return LAPATTN_ERR_HIP;
        }
        e = run_named(rec, "query_out", [&] {
            return lapattn::launch_query_out(LAPATTN_FP32, norm, q, out, at<float>(workspace, p.kt),
                                             at<float>(workspace, p.M), at<float>(workspace, p.Mc),
                                             at<float>(workspace, p.vbar), E,
                                             whiten_of(opts), at<float>(workspace, p.mvec),
                                             save ? at<float>(workspace, p.Aq) : nullptr, BH, H, n, d, m, lambda, st);
        });
        if (e != hipSuccess) return LAPATTN_ERR_HIP;
        if (bf16) {
            e = run_named(rec, "narrow", [&] {
                return lapattn::launch_narrow_bf16(at<float>(workspace, p.oF), nullptr, nullptr,
                                                   static_cast<uint16_t*>(Out), nullptr, nullptr, (size_t)BH * n * d,
                                                   st);
            });
        }
        return e == hipSuccess ? LAPATTN_OK : LAPATTN_ERR_HIP;
    } catch (...) {
        return LAPATTN_ERR_HIP;
    }
}

int lapattn_backward(const void* Q, const void* K, const void* V, const void* dOut, void* dQ, void* dK, void* dV,
                     int B, int H, int n, int d, int m, float lambda, int ns_iters, int dtype,
                     const lapattn_opts* opts, void* workspace, size_t workspace_bytes, lapattn_stream_t stream) {
    try {
        if (!Q || !K || !V || !dOut || !dQ || !dK || !dV) return LAPATTN_ERR_NULL;
        const int norm = norm_of(opts);
        const float eps = eps_of(opts);
        const lapattn::LmPool pl = pool_of(opts);
        const Dwc dwc = dwc_of(opts);
        int rc = check_shape(B, H, n, d, m, lambda, ns_iters, dtype, norm, eps);
        if (rc) return rc;
        if ((rc = check_pool(n, m, pl))) return rc;
        if ((rc = check_dwc(dwc, pl))) return rc;
        rc = check_align({Q, K, V, dOut, dQ, dK, dV}, workspace);
        if (rc) return rc;
        const int BH = B * H;
        const bool bf16 = dtype == LAPATTN_BF16;
        const Plan p = make_plan(BH, n, d, m, ns_iters, true, bf16, dwc.k != 0);
        if (!workspace || workspace_bytes < p.total) return LAPATTN_ERR_WORKSPACE;
        hipStream_t st = reinterpret_cast<hipStream_t>(stream);
        void* ws = workspace;
        Recorder rec(st);
        hipError_t e;
        // bf16 inputs: the backward runs in fp32 on the exact widened values, and the gradients
        // are rounded to bf16 at the end
        const size_t cnt = (size_t)BH * n * d;
        const float* q = bf16 ? at<float>(ws, p.wQ) : static_cast<const float*>(Q);
        const float* k = bf16 ? at<float>(ws, p.wK) : static_cast<const float*>(K);
        const float* v = bf16 ? at<float>(ws, p.wV) : static_cast<const float*>(V);
        const float* g = bf16 ? at<float>(ws, p.wG) : static_cast<const float*>(dOut);
        float* dq = bf16 ? at<float>(ws, p.gQ) : static_cast<float*>(dQ);
        float* dk = bf16 ? at<float>(ws, p.gK) : static_cast<float*>(dK);
        float* dv = bf16 ? at<float>(ws, p.gV) : static_cast<float*>(dV);
        if (bf16) {
            e = run_named(rec, "widen", [&] {
                return lapattn::launch_widen_bf16(static_cast<const uint16_t*>(Q), static_cast<const uint16_t*>(K),
                                                  static_cast<const uint16_t*>(V), static_cast<const uint16_t*>(dOut),
                                                  at<float>(ws, p.wQ), at<float>(ws, p.wK), at<float>(ws, p.wV),
                                                  at<float>(ws, p.wG), cnt, st);
            });
            if (e != hipSuccess) return LAPATTN_ERR_HIP;
        }
        // fp32 inputs with save: the forward left pool, key-side summary and solve (with every
        // iterate) in this workspace; otherwise they are recomputed here
        const bool saved = !bf16 && save_of(opts);
        if (!saved) {
            e = forward_internals(rec, p, q, k, v, ws, BH, n, d, m, lambda, ns_iters, LAPATTN_FP32, eps, true, pl,
                                  st);
            if (e != hipSuccess) return LAPATTN_ERR_HIP;
        }
        const bool mspace = norm == LAPATTN_NORM_MSPACE;
        const float* whiten = whiten_of(opts);
        if (mspace) {
            e = run_named(rec, "mspace_vec", [&] {
                return lapattn::launch_mspace_vec(at<float>(ws, p.M), whiten, at<float>(ws, p.mvec), BH, H, d, m, st);
            });
            if (e != hipSuccess) return LAPATTN_ERR_HIP;
        }
        e = run_named(rec, "bwd_query", [&] {
            return lapattn::launch_bwd_query(norm, q, g, dq, at<float>(ws, p.kt), at<float>(ws, p.M),
                                             at<float>(ws, p.vbar), at<float>(ws, p.Aq), at<float>(ws, p.dDq),
                                             at<float>(ws, p.rs), at<float>(ws, p.dYd), at<float>(ws, p.dvbar_part),
                                             at<float>(ws, p.p0_part), whiten, at<float>(ws, p.mvec), saved ? 1 : 0, BH,
                                             H, n, d, m, lambda, p.nqb, st);
        });
        if (e != hipSuccess) return LAPATTN_ERR_HIP;
        e = run_named(rec, "bwd_query_lm", [&] {
            return lapattn::launch_bwd_query_lm(q, g, at<float>(ws, p.kt), at<float>(ws, p.Aq), at<float>(ws, p.dDq),
                                                at<float>(ws, p.rs), at<float>(ws, p.dYd), at<float>(ws, p.dM_part),
                                                at<float>(ws, p.dkt_part), BH, n, d, m, p.lmc, p.nlc, st);
        });
        if (e != hipSuccess) return LAPATTN_ERR_HIP;
        if (p.MP == 128)
            e = run_named(rec, "bwd_ns", [&] {
                return lapattn::launch_nsb_backward(
                    at<float>(ws, p.qt), at<float>(ws, p.kt), at<double>(ws, p.Xs), at<double>(ws, p.cinfo),
                    at<float>(ws, p.U), at<float>(ws, p.dM_part), at<float>(ws, p.dvbar_part), at<float>(ws, p.p0_part),
                    whiten, mspace ? 1 : 0, at<float>(ws, p.dU), at<float>(ws, p.dvbar), at<float>(ws, p.dqtW),
                    at<float>(ws, p.dkpool), at<float>(ws, p.dkt_part), pl, at<double>(ws, p.nsbs), at<float>(ws, p.dDW),
                    BH, H, n, d, m, ns_iters, (double)lambda, (double)eps, p.nlc, p.nqb, st);
            });
        else
        e = run_named(rec, "bwd_ns", [&] {
            return lapattn::launch_bwd_ns(at<float>(ws, p.qt), at<float>(ws, p.kt), at<double>(ws, p.Xs),
                                          at<double>(ws, p.cinfo), at<float>(ws, p.U), at<float>(ws, p.dM_part),
                                          at<float>(ws, p.dvbar_part), at<float>(ws, p.dU), at<float>(ws, p.dvbar),
                                          at<float>(ws, p.dqtW), at<float>(ws, p.dkpool), at<float>(ws, p.dkt_part), pl,
                                          at<float>(ws, p.p0_part), whiten, mspace ? 1 : 0, at<float>(ws, p.dDW), BH,
                                          H, n, d, m, ns_iters,
                                          (double)lambda,
                                          (double)eps, p.nlc, p.nqb, p.MP, st);
        });
        if (e != hipSuccess) return LAPATTN_ERR_HIP;
        e = run_named(rec, "bwd_key", [&] {
            return lapattn::launch_bwd_key(k, v, dk, dv, at<float>(ws, p.qt), at<float>(ws, p.dU),
                                           at<float>(ws, p.dvbar), at<float>(ws, p.dDk), at<float>(ws, p.dkpool), pl,
                                           saved ? 1 : 0, BH, n, d, m, lambda, st);
        });
        if (e != hipSuccess) return LAPATTN_ERR_HIP;
        e = run_named(rec, "bwd_key_lm", [&] {
            return lapattn::launch_bwd_key_lm(k, at<float>(ws, p.qt), at<float>(ws, p.dDk), at<float>(ws, p.dqt_part),
                                              BH, n, d, m, p.lmc, p.nlc, st);
        });
        if (e != hipSuccess) return LAPATTN_ERR_HIP;
        e = run_named(rec, "bwd_pool", [&] {
            return lapattn::launch_bwd_pool(dq, at<float>(ws, p.dqtW), at<float>(ws, p.dqt_part), BH, n, d, m, p.nlc,
                                            pl, st);
        });
        if (e != hipSuccess) return LAPATTN_ERR_HIP;
        if (dwc.k) {
            e = run_named(rec, "dwc_dv", [&] {
                return lapattn::launch_dwc_bwd_dv(g, dwc.w, dv, BH, H, n, d, pl.gw, dwc.k, st);
            });
            if (e != hipSuccess) return LAPATTN_ERR_HIP;
            if (dwc.dw || dwc.db) {
                e = run_named(rec, "dwc_dw", [&] {
                    return lapattn::launch_dwc_bwd_w(g, v, at<float>(ws, p.dwc_part), dwc.dw, dwc.db, B, H, n, d,
                                                     pl.gw, dwc.k, kDwcChunk, st);
                });
                if (e != hipSuccess) return LAPATTN_ERR_HIP;
            }
        }
        if (!bf16) return LAPATTN_OK;
        e = run_named(rec, "narrow", [&] {
            return lapattn::launch_narrow_bf16(dq, dk, dv, static_cast<uint16_t*>(dQ), static_cast<uint16_t*>(dK),
                                               static_cast<uint16_t*>(dV), cnt, st);
        });
        return e == hipSuccess ? LAPATTN_OK : LAPATTN_ERR_HIP;
    } catch (...) {
        return LAPATTN_ERR_HIP;
    }
}

const char* lapattn_status_str(int status) {
    switch (status) {
        case LAPATTN_OK: return "ok";
        case LAPATTN_ERR_NULL: return "null pointer argument";
        case LAPATTN_ERR_SHAPE: return "invalid shape (B, H, n >= 1, 1 <= m <= n, B*H*n*d < 2^31)";
        case LAPATTN_ERR_PARAM:
            return "invalid parameter (lambda, ns_iters, eps, norm, dtype, map or convolution options)";
        case LAPATTN_ERR_UNSUPPORTED: return "unsupported configuration (d in {32, 64}, m <= 128)";
        case LAPATTN_ERR_WORKSPACE: return "workspace missing or too small";
        case LAPATTN_ERR_HIP: return "HIP launch failed";
        case LAPATTN_ERR_ALIGN: return "a tensor is not 16-byte aligned or the workspace not 256-byte aligned";
        case LAPATTN_ERR_SCRATCH: return "the call needs more workspace than the static scratch array holds (32 MiB)";
        default: return "unknown status";
    }
}

int lapattn_timing_enable(int enable) {
    Timing& t = timing();
    std::lock_guard<std::mutex> g(t.mu);
    int prev = t.enabled ? 1 : 0;
    t.enabled = enable != 0;
    if (t.enabled) {
        t.names.clear();
        t.used = 0;
    }
    return prev;
}

int lapattn_timing_read(float* ms, int cap) {
    Timing& t = timing();
    std::lock_guard<std::mutex> g(t.mu);
    const int nk = (int)t.names.size();
    for (int i = 0; i < nk && i < cap && ms; ++i) {
        if (hipEventSynchronize(t.ev[2 * i + 1]) != hipSuccess) return -1;
        float v = 0.f;
        if (hipEventElapsedTime(&v, t.ev[2 * i], t.ev[2 * i + 1]) != hipSuccess) return -1;
        ms[i] = v;
    }
    return nk;
}

const char* lapattn_timing_name(int index) {
    Timing& t = timing();
    std::lock_guard<std::mutex> g(t.mu);
    if (index < 0 || index >= (int)t.names.size()) return "";
    return t.names[index];
}

}  // extern "C"
