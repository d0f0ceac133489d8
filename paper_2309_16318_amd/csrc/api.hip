// Host side of the DeepPCR C ABI: argument validation (before any HIP call),
// workspace carving, the PCR level loop and the Newton driver.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <atomic>
#include <chrono>
#include <mutex>
#include <vector>

#include "../../include/deeppcr.h"
#include "internal.h"

using namespace deeppcr;

namespace {

thread_local char g_last_error[256] = "";

int hip_fail(hipError_t e, const char* where) {
    std::snprintf(g_last_error, sizeof g_last_error, "%s: %s (%d)", where, hipGetErrorString(e),
                  (int)e);
    return DEEPPCR_EHIP;
}

#define DEEPPCR_HIP(call)                                  \
    do {                                                   \
        hipError_t e_ = (call);                            \
        if (e_ != hipSuccess) return hip_fail(e_, #call);  \
    } while (0)

// ------------------------------------------------------------ instrumentation
// One record per span: consecutive launches of one kernel class on one
// stream, with nothing else enqueued in between, share one event pair, so
// that short kernels are not charged the cost of an event pair each.  The
// end event is recorded when the span ends (the next launch of another
// class, any other enqueue of the library, or the return of an entry point),
// so that no event sits between the kernels of a span.
struct ProfRec {
    int kclass;
    hipStream_t st;
    hipEvent_t e0, e1;
    long long n;
    double bytes, flops;
    bool share0;  // e0 is the end event of the record before (owned there)
};

// Per host thread: the instrumentation of a thread sees only the launches
// that thread makes (enable, select, reset and read act on the calling
// thread's state).
struct Prof {
    bool on = false;
    unsigned mask = ~0u;  // classes that are timed
    bool open = false;  // the last record may be extended; its end event is not recorded yet
    std::vector<ProfRec> pending;
    std::vector<hipEvent_t> pool;
    long long launches[DEEPPCR_KCLASS_COUNT] = {};
    double ms[DEEPPCR_KCLASS_COUNT] = {};
    double bytes[DEEPPCR_KCLASS_COUNT] = {};
    double flops[DEEPPCR_KCLASS_COUNT] = {};
};
thread_local Prof g_prof;

hipEvent_t take_event() {
    if (!g_prof.pool.empty()) {
        hipEvent_t e = g_prof.pool.back();
        g_prof.pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Ends the current span: its end event is recorded now, right behind its
// last launch.  Called before every enqueue that is not a timed launch and
// when an entry point returns.
hipError_t prof_break() {
    if (!g_prof.open) return hipSuccess;
    g_prof.open = false;
    const ProfRec& r = g_prof.pending.back();
    return hipEventRecord(r.e1, r.st);
}

// Ends the span at every exit of an entry point.
struct SpanGuard {
    SpanGuard() { (void)prof_break(); }
    ~SpanGuard() { (void)prof_break(); }
    SpanGuard(const SpanGuard&) = delete;
    SpanGuard& operator=(const SpanGuard&) = delete;
};

// Runs `launch` (which enqueues one kernel on `st` and returns its
// hipGetLastError), bracketed by events when instrumentation is on.
// A launch of a class that is not timed ends the open span first.  Where a
// span of another class on the same stream is open, one event ends it and
// starts the new one (each event is a marker between two kernels, which
// costs the stream a few microseconds).
template <class F>
hipError_t timed(int kclass, double bytes, double flops, hipStream_t st, F&& launch) {
    if (!g_prof.on) return launch();
    if (!((g_prof.mask >> kclass) & 1u)) {
        hipError_t e = prof_break();
        if (e != hipSuccess) return e;
        return launch();
    }
    if (g_prof.open) {
        ProfRec& r = g_prof.pending.back();
        if (r.kclass == kclass && r.st == st) {
            hipError_t e = launch();
            if (e != hipSuccess) return e;
            r.n += 1;
            r.bytes += bytes;
            r.flops += flops;
            return hipSuccess;
        }
        if (r.st == st) {
            hipEvent_t e1 = take_event();
            if (e1) {
                const hipEvent_t e0 = r.e1;
                g_prof.open = false;
                hipError_t e = hipEventRecord(e0, st);
                if (e != hipSuccess) return e;
                e = launch();
                if (e != hipSuccess) return e;
                g_prof.pending.push_back({kclass, st, e0, e1, 1, bytes, flops, true});
                g_prof.open = true;
                return hipSuccess;
            }
        }
        hipError_t e = prof_break();
        if (e != hipSuccess) return e;
    }
    hipEvent_t e0 = take_event(), e1 = take_event();
    if (!e0 || !e1) {
        // no event pair: run untimed and keep whichever event was obtained
        if (e0) g_prof.pool.push_back(e0);
        if (e1) g_prof.pool.push_back(e1);
        return launch();
    }
    hipError_t e = hipEventRecord(e0, st);
    if (e != hipSuccess) return e;
    e = launch();
    if (e != hipSuccess) return e;
    g_prof.pending.push_back({kclass, st, e0, e1, 1, bytes, flops, false});
    g_prof.open = true;
    return hipSuccess;
}

// An asynchronous copy on the stream (ending the instrumentation span).
hipError_t copy_async(void* dst, const void* src, size_t n, hipMemcpyKind kind, hipStream_t st) {
    hipError_t e = prof_break();
    if (e != hipSuccess) return e;
    return hipMemcpyAsync(dst, src, n, kind, st);
}

// Waits for the stream (ending the instrumentation span).
hipError_t host_wait(hipStream_t st) {
    hipError_t e = prof_break();
    if (e != hipSuccess) return e;
    return hipStreamSynchronize(st);
}

// ------------------------------------------------------------------ sizes
constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
    size_t A[2], r[2], dscale, red, total;
};

bool sizes_ok(int B, int L, int w) {
    return B >= 1 && L >= 1 && w >= 1 && w <= DEEPPCR_MAX_WIDTH &&
           (double)B * L * w * w * 4.0 * 2.0 < 9.0e18;
}

Layout layout(int op, int B, int L, int w) {
    const size_t nA = (size_t)B * L * w * w * sizeof(float);
    const size_t nr = (size_t)B * L * w * sizeof(float);
    Layout lo{};
    size_t off = 0;
    lo.A[0] = off; off += align_up(nA);
    lo.A[1] = off; off += align_up(nA);
    lo.r[0] = off; off += align_up(nr);
    lo.r[1] = off; off += align_up(nr);
    lo.dscale = off;
    if (op == DEEPPCR_OP_BWD) off += align_up(nr);
    lo.red = off; off += align_up(kRedWords * sizeof(unsigned));
    lo.total = off;
    return lo;
}

// Collapsed-skip ResNet: the block chain has G = L / skip rows; the forward
// keeps its iterate X [B, G, w] in the slot of the backward's c*d vectors.
Layout resnet_layout(int op, int B, int G, int w) {
    const size_t nA = (size_t)B * G * w * w * sizeof(float);
    const size_t nr = (size_t)B * G * w * sizeof(float);
    Layout lo{};
    size_t off = 0;
    lo.A[0] = off; off += align_up(nA);
    lo.A[1] = off; off += align_up(nA);
    lo.r[0] = off; off += align_up(nr);
    lo.r[1] = off; off += align_up(nr);
    lo.dscale = off;
    if (op == DEEPPCR_OP_FWD) off += align_up(nr);
    lo.red = off; off += align_up(kRedWords * sizeof(unsigned));
    lo.total = off;
    return lo;
}

// The ResNet block kernels and the chunked solve hold a whole block per
// workgroup: widths up to DEEPPCR_MAX_BLOCK_WIDTH.
bool block_sizes_ok(int B, int L, int w) { return sizes_ok(B, L, w) && w <= DEEPPCR_MAX_BLOCK_WIDTH; }

bool resnet_shape_ok(int B, int L, int w, int skip, int act) {
    return block_sizes_ok(B, L, w) && skip >= 1 && L % skip == 0 && act >= 0 && act <= 2;
}

int num_levels(int L) {
    int k = 0;
    for (long long s = 1; s < L; s *= 2) ++k;
    return k;
}

// Kernel launches of a PCR sweep: pairs of levels where the width has the
// two-level kernel, plus a single last level when the level count is odd.
int num_passes(int B, int L, int w) {
    const int kt = tail_levels(B, L, w, 0);
    const int K1 = num_levels(L) - kt;
    return (two_level(B, L, w) ? (K1 + 1) / 2 : K1) + (kt > 0 ? 1 : 0);
}

// Every array argument must start on a 16-byte boundary (the kernels load
// rows of blocks, states and weights as 16-byte vectors); NULL passes (the
// null checks are separate).
bool aligned(std::initializer_list<const void*> ps) {
    for (const void* p : ps)
        if (((uintptr_t)p & 15u) != 0) return false;
    return true;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    if (!a || !b || na == 0 || nb == 0) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + nb && b0 < a0 + na;
}

// Algorithmic work of one PCR level at stride s over B systems: (L-s) mat-vecs
// and (L-2s)+ block products per system; bytes = A_l reads for l >= s, A writes
// for l >= 2s, one read and one write of every r row.
void level_work(int B, int L, int w, int s, double* bytes, double* flops) {
    const double nr = (double)(L - s), na = (double)(L - 2 * s > 0 ? L - 2 * s : 0);
    const double w2 = (double)w * w;
    *bytes = 4.0 * B * (nr * w2 + na * w2 + 2.0 * L * w);
    *flops = (double)B * (nr * 2.0 * w2 + na * 2.0 * w2 * w);
}

// Algorithmic work of a fused pair of levels (strides s, 2s): the flops of
// both levels; the bytes the fused pass must move: A_l read for l >= s, the
// level-2s operators written for l >= 4s, r read and written once.
void level2_work(int B, int L, int w, int s, double* bytes, double* flops) {
    double b1, f1, b2, f2;
    level_work(B, L, w, s, &b1, &f1);
    level_work(B, L, w, 2 * s, &b2, &f2);
    const double nr = (double)(L - s), na = (double)(L - 4 * s > 0 ? L - 4 * s : 0);
    const double w2 = (double)w * w;
    *bytes = 4.0 * B * (nr * w2 + na * w2 + 2.0 * L * w);
    *flops = f1 + f2;
}

// Algorithmic work of the last two levels as mat-vecs only (strides s, 2s,
// 4s >= L): A_l read once for l >= s; mat-vecs A_l r_{l-s} and
// A_l r'_{l-s} for l >= s, A_l t_{l-s} for l >= 2s; r read and written once.
void last2_work(int B, int L, int w, int s, double* bytes, double* flops) {
    const double n1 = (double)(L - s), n2 = (double)(L - 2 * s > 0 ? L - 2 * s : 0);
    const double w2 = (double)w * w;
    *bytes = 4.0 * B * (n1 * w2 + 2.0 * L * w);
    *flops = (double)B * 2.0 * w2 * (2.0 * n1 + n2);
}

// Algorithmic work of the last kt levels solved by substitution along the
// chains (s = 2^(levels - kt)): A_l read once and one mat-vec for every row
// l >= s; r read and the solution written.
void tail_work(int B, int L, int w, int kt, double* bytes, double* flops) {
    const int s = 1 << (num_levels(L) - kt);
    const double w2 = (double)w * w;
    *bytes = 4.0 * B * ((double)(L - s) * w2 + 2.0 * L * w);
    *flops = (double)B * (L - s) * 2.0 * w2;
}

// Stride of the rows the last kt levels start from.
int tail_stride(int L, int kt) { return 1 << (num_levels(L) - kt); }

// Runs all PCR levels.  Level 0 reads (A0, r0); level k writes operators to
// ws A buffer (k + a_first) % 2 and vectors to ws r buffer (k + r_first) % 2,
// except the last level, which writes the solution to `x`.
// With bwd the first pass (levels 1 and 2) forms the backward's blocks from
// the weights instead of reading A0 (w = 32, 64, 128 and L > 2 only).
hipError_t pcr_sweep(const BlockSrc& A0, const VecSrc& r0, const VecDst& x, int B, int L, int w,
                     float* wsA[2], float* wsr[2], int a_first, int r_first, hipStream_t st,
                     const BwdArgs* bwd = nullptr, unsigned* upd_red = nullptr) {
    const int K = num_levels(L);
    if (K == 0) {
        const double bytes = 8.0 * B * L * w;
        return timed(DEEPPCR_KCLASS_OTHER, bytes, 0.0, st,
                     [&] { return launch_copy_rows(r0, x, B, L, w, st); });
    }
    const bool two = two_level(B, L, w);
    const int kt = tail_levels(B, L, w, 0);
    const int K1 = K - kt;  // levels before the tail
    BlockSrc Ain = A0;
    VecSrc rin = r0;
    int s = 1;
    // pass p writes operators to ws A buffer (p + a_first) % 2 and vectors to
    // ws r buffer (p + r_first) % 2; the last pass writes the solution to x
    // (the tail pass, when there is one, after the levels below K1)
    const int Kend = kt > 0 ? K1 : K;
    for (int k = 0, p = 0; k < Kend; ++p) {
        const bool pair = two && k + 1 < Kend;
        const bool last = kt == 0 && (k + (pair ? 1 : 0)) == K - 1;
        float* Aout = wsA[(p + a_first) & 1];
        VecDst rout = last ? x
                           : VecDst{wsr[(p + r_first) & 1], (long long)L * w, (long long)w};
        double bytes, flops;
        hipError_t e;
        if (bwd && k == 0) {
            // blocks from the weights (read from L2): the products and r
            level2_work(B, L, w, s, &bytes, &flops);
            bytes -= 4.0 * B * (L - 1) * (double)w * w;
            e = timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st, [&] {
                return launch_pcr_level2_bwd(*bwd, rin, Aout, rout, B, L, w, st);
            });
        } else if (pair && last && last_pair_width(w)) {
            last2_work(B, L, w, s, &bytes, &flops);
            e = timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st, [&] {
                return launch_pcr_level2_last(Ain, rin, rout, B, L, w, s, st);
            });
        } else if (pair) {
            level2_work(B, L, w, s, &bytes, &flops);
            e = timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st, [&] {
                return launch_pcr_level2(Ain, rin, Aout, rout, B, L, w, s, st);
            });
        } else {
            level_work(B, L, w, s, &bytes, &flops);
            e = timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st, [&] {
                return wide_width(w) ? launch_pcr_level_wide(Ain, rin, Aout, rout, B, L, w, s, st)
                                     : launch_pcr_level(Ain, rin, Aout, rout, B, L, w, s, st);
            });
        }
        if (e != hipSuccess) return e;
        Ain = BlockSrc{Aout, (long long)L * w * w, (long long)w * w, 0};
        rin = VecSrc{rout.base, rout.bstride, rout.rstride};
        s *= pair ? 4 : 2;
        k += pair ? 2 : 1;
    }
    if (kt == 0) return hipSuccess;
    double bytes, flops;
    tail_work(B, L, w, kt, &bytes, &flops);
    if (upd_red) bytes += 4.0 * B * L * w;  // the iterate is read as well
    return timed(DEEPPCR_KCLASS_PCR_TAIL, bytes, flops, st, [&] {
        return launch_pcr_chain_subst(Ain, rin, x, B, L, w, tail_stride(L, kt), st, upd_red);
    });
}

struct Ws {
    float* A[2];
    float* r[2];
    float* dscale;
    unsigned* red;
};

Ws carve(void* workspace, const Layout& lo) {
    char* p = (char*)workspace;
    Ws ws;
    ws.A[0] = (float*)(p + lo.A[0]);
    ws.A[1] = (float*)(p + lo.A[1]);
    ws.r[0] = (float*)(p + lo.r[0]);
    ws.r[1] = (float*)(p + lo.r[1]);
    ws.dscale = (float*)(p + lo.dscale);
    ws.red = (unsigned*)(p + lo.red);
    return ws;
}

// Pinned, mapped host words that kernels write the per-call and
// per-iteration records into: words 0-3 the one-launch solver's status
// record and completion word, words 4-7 (kHostMeas) the Newton measures and
// their sequence word.  Allocated on the first Newton call of a host thread;
// deeppcr_release_thread_state frees them.
constexpr int kHostMeas = 4, kHostWords = 8;
thread_local unsigned* g_host_words = nullptr;

unsigned* host_words() {
    if (!g_host_words) {
        void* p = nullptr;
        if (hipHostMalloc(&p, kHostWords * sizeof(unsigned),
                          hipHostMallocMapped | hipHostMallocPortable) != hipSuccess)
            return nullptr;
        std::memset(p, 0, kHostWords * sizeof(unsigned));
        g_host_words = (unsigned*)p;
    }
    return g_host_words;
}

float bits_to_float(unsigned u) {
    float f;
    std::memcpy(&f, &u, sizeof f);
    return f;
}

// Waits until the host-mapped word `word`, which a kernel writes after its
// record, holds `value`: the host watches it for up to 5 ms (Newton
// iterations and small solves take microseconds to a few milliseconds) and
// then waits for the stream, which also reports a failed launch.  The
// acquire fence orders the record's reads after the word's.
hipError_t watch_word(const volatile unsigned* word, unsigned value, hipStream_t st) {
    hipError_t e = prof_break();
    if (e != hipSuccess) return e;
    bool seen = false;
    const auto t0 = std::chrono::steady_clock::now();
    while (!(seen = (*word == value)) &&
           std::chrono::steady_clock::now() - t0 < std::chrono::milliseconds(5)) {
    }
    if (!seen) {
        e = host_wait(st);
        if (e != hipSuccess) return e;
        if (*word != value) return hipErrorUnknown;
    }
    std::atomic_thread_fence(std::memory_order_acquire);
    return hipSuccess;
}

// The stopping measures of a Newton iteration, after its last kernel on st:
// m[0] = max |dZ|, m[1] = max |Z|, m[2] = max |F| (float bit patterns, the
// max over each measure's slots of red).  One small kernel reduces the slots
// and writes them with a fresh sequence number into the host words, which
// the host watches instead of waiting for the stream.
hipError_t read_measures(const unsigned* red, unsigned* hw, hipStream_t st, unsigned m[3]) {
    thread_local unsigned seq = 0u;
    seq = seq + 1u == 0u ? 1u : seq + 1u;
    void* hwd = nullptr;
    hipError_t e = hipHostGetDevicePointer(&hwd, hw, 0);
    if (e != hipSuccess) return e;
    e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * kRedWords, 0.0, st, [&] {
        return launch_measures(red, (unsigned*)hwd + kHostMeas, seq, st);
    });
    if (e != hipSuccess) return e;
    const volatile unsigned* rec = hw + kHostMeas;
    e = watch_word(rec + 3, seq, st);
    if (e != hipSuccess) return e;
    for (int j = 0; j < 3; ++j) m[j] = rec[j];
    return hipSuccess;
}

// The fused Newton linear solve (w = 16, 32, 64, 128): the layer evaluation
// runs inside the first PCR pass (level 1, or levels 1 and 2 where
// first_level_count says so); for w = 16, 32 without a tail pass the update
// + reduction runs inside the last level, otherwise the last pass writes the
// solution (as does the first for L <= 2, to `x`) and the separate update
// kernel applies it.
// Split in two so that a stopping test on the residual (reduced by the first
// level) can sit between the halves.
hipError_t fused_first_level(const NewtonArgs& na, int B, int L, int w, const Ws& ws,
                             const VecDst& x, hipStream_t st) {
    const int K = num_levels(L);
    const double w2 = (double)w * w;
    const long long ld = (long long)L * w;
    // the first level (or two) with the layers: W once, Z read twice,
    // products and r written
    const int nl = first_level_count(B, L, w);
    const double na2 = (double)(L - 2 * nl > 0 ? L - 2 * nl : 0);
    const double bytes = 4.0 * ((double)L * w2 + B * (na2 * w2 + 3.0 * L * w));
    double flops = (double)B * (L * 3.0 * w2 + (L - 1) * 2.0 * w2 +
                                (L - 2 > 0 ? L - 2 : 0) * 2.0 * w2 * w);
    if (nl == 2) {
        double b2, f2;
        level_work(B, L, w, 2, &b2, &f2);
        flops += f2;
    }
    const VecDst out = (K <= 1) ? x : VecDst{ws.r[0], ld, (long long)w};
    return timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st,
                 [&] { return launch_first_level_fwd(na, ws.A[0], out, B, L, w, st); });
}

hipError_t fused_rest_levels(const NewtonArgs& na, int B, int L, int w, const Ws& ws,
                             const VecDst& x, hipStream_t st) {
    const int K = num_levels(L);
    const long long ld = (long long)L * w;
    if (K <= 1) {
        const long long n = (long long)B * L * w;
        return timed(DEEPPCR_KCLASS_UPDATE, 12.0 * n, 2.0 * n, st,
                     [&] { return launch_update_reduce(na.Z, x.base, n, na.red, st); });
    }
    // the last levels go to one tail pass where tail_levels says so; else for
    // w = 16, 32 the last level applies the update itself
    const int k0 = first_level_count(B, L, w);
    const int kt = tail_levels(B, L, w, k0);
    const bool upd = fused_newton_levels(w) && kt == 0 && k0 < K;
    const int Kp = upd ? K - 1 : K - kt;
    BlockSrc Ain{ws.A[0], (long long)L * w * w, (long long)w * w, 0};
    VecSrc rin{ws.r[0], ld, (long long)w};
    // the levels after the first one (or two) up to Kp-1, two per pass where
    // possible; pass p writes ws buffers p % 2 (the first pass wrote buffers 0)
    int s = 1 << k0, p = 1;
    for (int k = k0; k < Kp; ++p) {
        const bool pair = two_level(B, L, w) && k + 1 < Kp;
        float* Aout = ws.A[p & 1];
        const VecDst rout{ws.r[p & 1], ld, (long long)w};
        double bytes, flops;
        hipError_t e;
        if (pair && !upd && kt == 0 && k + 1 == K - 1 && last_pair_width(w)) {
            last2_work(B, L, w, s, &bytes, &flops);
            e = timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st, [&] {
                return launch_pcr_level2_last(Ain, rin, rout, B, L, w, s, st);
            });
        } else if (pair) {
            level2_work(B, L, w, s, &bytes, &flops);
            e = timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st, [&] {
                return launch_pcr_level2(Ain, rin, Aout, rout, B, L, w, s, st);
            });
        } else {
            level_work(B, L, w, s, &bytes, &flops);
            e = timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st, [&] {
                return launch_pcr_level(Ain, rin, Aout, rout, B, L, w, s, st);
            });
        }
        if (e != hipSuccess) return e;
        Ain = BlockSrc{Aout, (long long)L * w * w, (long long)w * w, 0};
        rin = VecSrc{rout.base, rout.bstride, rout.rstride};
        s *= pair ? 4 : 2;
        k += pair ? 2 : 1;
    }
    if (kt > 0) {
        // the chains left for the last kt levels solved by substitution in
        // one pass, which also applies the update Z += x and reduces the
        // convergence maxima (the iterate is read and written instead of
        // the solution being written)
        double bytes, flops;
        tail_work(B, L, w, kt, &bytes, &flops);
        bytes += 4.0 * B * L * w;
        const VecDst zo{na.Z, ld, (long long)w};
        return timed(DEEPPCR_KCLASS_PCR_TAIL, bytes, flops, st, [&] {
            return launch_pcr_chain_subst(Ain, rin, zo, B, L, w, tail_stride(L, kt), st,
                                          na.red);
        });
    }
    if (!upd) {
        // the last pass wrote the solution to the ws r buffer rin reads
        const long long n = (long long)B * L * w;
        return timed(DEEPPCR_KCLASS_UPDATE, 12.0 * n, 2.0 * n, st,
                     [&] { return launch_update_reduce(na.Z, rin.base, n, na.red, st); });
    }
    // the last level with the update Z += x and the convergence reduction
    double bytes, flops;
    level_work(B, L, w, s, &bytes, &flops);
    bytes += 8.0 * B * L * w;  // the iterate is read and written
    return timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st, [&] {
        return launch_last_level_update(Ain, rin, na, B, L, w, s, st);
    });
}

// Argument checks shared by the two forward entry points.
int check_forward_args(const float* W, const float* bias, const float* z0, float* Z,
                       const float* Z_init, void* workspace, size_t workspace_bytes, int B,
                       int L, int w, int layer, float alpha) {
    if (!W || !bias || !z0 || !Z || !workspace || !sizes_ok(B, L, w)) return DEEPPCR_EINVAL;
    if (layer < 0 || layer >= kNumLayerKinds || !std::isfinite(alpha)) return DEEPPCR_EINVAL;
    if (!aligned({W, bias, z0, Z, Z_init, workspace})) return DEEPPCR_EINVAL;
    const Layout lo = layout(DEEPPCR_OP_FWD, B, L, w);
    if (workspace_bytes < lo.total) return DEEPPCR_EWORKSPACE;
    const size_t nv = (size_t)B * L * w * 4;
    if (overlaps(workspace, lo.total, Z, nv) ||
        overlaps(workspace, lo.total, W, (size_t)L * w * w * 4) ||
        overlaps(workspace, lo.total, z0, (size_t)B * w * 4) ||
        overlaps(workspace, lo.total, bias, (size_t)L * w * 4) ||
        overlaps(workspace, lo.total, Z_init, Z_init ? nv : 0))
        return DEEPPCR_EINVAL;
    if (Z_init && Z_init != Z && overlaps(Z_init, nv, Z, nv)) return DEEPPCR_EINVAL;
    return DEEPPCR_OK;
}

// The Newton driver behind both forward entry points (Sec. 2, Eqs. 1-3).
// Update rule: up to max_iter solves, each followed by the update and the
// test max|dZ| < tol * max(1, max|Z|) (tol = 0: exactly max_iter solves).
// Residual rule: for k = 0..max_iter the residual F(z^k) is reduced while
// the layers are evaluated, and the iteration stops before the solve when
// max|F| <= atol or max|F| <= rtol * max|F(z^0)|.  One host read-back per
// iteration either way.  *measure_out = the last max|dZ| or max|F|.
int newton_forward(const float* W, const float* bias, const float* z0, float* Z, int B, int L,
                   int w, int layer, float alpha, const StopRule& rule, const float* Z_init,
                   void* workspace, int* iters_out, float* measure_out, hipStream_t st) {
    const Layout lo = layout(DEEPPCR_OP_FWD, B, L, w);
    const size_t nv = (size_t)B * L * w * 4;
    Ws ws = carve(workspace, lo);
    unsigned* hw = host_words();
    if (!hw) return hip_fail(hipErrorOutOfMemory, "hipHostMalloc");
    if (iters_out) *iters_out = 0;
    if (measure_out) *measure_out = 0.f;

    if (tiny_eligible(B, L, w)) {
        // one launch for the whole solve; reads W, bias, z0 (and Z_init), writes Z
        // and its status record straight into the mapped host words
        void* hwd = nullptr;
        DEEPPCR_HIP(hipHostGetDevicePointer(&hwd, hw, 0));
        const double io = 4.0 * ((double)L * w * (w + 1) + B * w + 2.0 * B * L * w);
        // the kernel writes the status record, then hw[3] = 1: the host
        // watches that word (for up to 5 ms, against solves of 10-30 us) and
        // waits for the stream only if it does not arrive
        volatile unsigned* done = hw + 3;
        *done = 0u;
        hipError_t e = timed(DEEPPCR_KCLASS_PCR_LEVEL, io, 0.0, st, [&] {
            return launch_newton_tiny(W, bias, z0, Z, Z_init, B, L, w, layer, alpha, rule,
                                      (unsigned*)hwd, st);
        });
        if (e != hipSuccess) return hip_fail(e, "newton_tiny");
        DEEPPCR_HIP(watch_word(done, 1u, st));
        if (iters_out) *iters_out = (int)hw[1];
        if (measure_out) *measure_out = bits_to_float(hw[2]);
        if (hw[0] == 3u) return DEEPPCR_ENONFINITE;
        if (hw[0] == 2u) return DEEPPCR_ENOCONV;
        return DEEPPCR_OK;
    }
    const double w2 = (double)w * w;
    const double eval_bytes = 4.0 * B * L * (w2 + 2.0 * w);
    const double eval_flops = (double)B * L * (2.0 * w2 + w2);
    if (Z_init) {
        if (Z_init != Z) DEEPPCR_HIP(copy_async(Z, Z_init, nv, hipMemcpyDeviceToDevice, st));
    } else {
        hipError_t e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * B * L * w, 2.0 * B * w * w, st, [&] {
            return launch_initial_guess(W, bias, z0, Z, B, L, w, layer, alpha, st);
        });
        if (e != hipSuccess) return hip_fail(e, "initial_guess");
    }
    const long long n = (long long)B * L * w;
    const VecDst xd{ws.r[(num_passes(B, L, w) + 1) & 1], (long long)L * w, (long long)w};
    const bool fused = layer_first_level(w);
    const NewtonArgs na{W, bias, z0, Z, ws.red, layer, alpha};
    unsigned* fslots = ws.red + kRedF;
    if (rule.residual) {
        hipError_t e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * kRedShards, 0.0, st,
                             [&] { return launch_zero_words(fslots, kRedShards, st); });
        if (e != hipSuccess) return hip_fail(e, "zero_words");
    }
    float res0 = 0.f;
    for (int k = 0; k <= rule.max_iter; ++k) {
        if (!rule.residual && k == rule.max_iter) break;
        // Layers, Jacobian blocks (forward order) and residuals at the iterate:
        // fused into the first PCR level, or evaluated into ws A[1], r[1].
        hipError_t e;
        if (fused) {
            e = fused_first_level(na, B, L, w, ws, xd, st);
        } else {
            e = timed(DEEPPCR_KCLASS_LAYER, eval_bytes, eval_flops, st, [&] {
                return launch_forward_eval(W, bias, z0, Z, ws.A[1], ws.r[1], ws.red, B, L, w,
                                           layer, alpha, st);
            });
        }
        if (e != hipSuccess) return hip_fail(e, "layer evaluation");
        if (rule.residual) {
            unsigned ms[3];
            DEEPPCR_HIP(read_measures(ws.red, hw, st, ms));
            const unsigned mf = ms[2];
            if (iters_out) *iters_out = k;
            if (measure_out) *measure_out = bits_to_float(mf);
            if (mf >= 0x7f800000u) return DEEPPCR_ENONFINITE;
            const float res = bits_to_float(mf);
            if (k == 0) res0 = res;
            if (res <= rule.atol || res <= rule.rtol * res0) return DEEPPCR_OK;
            if (k == rule.max_iter) return DEEPPCR_ENOCONV;
            e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * kRedShards, 0.0, st,
                      [&] { return launch_zero_words(fslots, kRedShards, st); });
            if (e != hipSuccess) return hip_fail(e, "zero_words");
        }
        // The rest of the solve of Eq. 3 and the update Z += dZ.
        if (fused) {
            e = fused_rest_levels(na, B, L, w, ws, xd, st);
            if (e != hipSuccess) return hip_fail(e, "newton levels");
        } else {
            e = pcr_sweep(BlockSrc{ws.A[1], (long long)L * w * w, (long long)w * w, 0},
                          VecSrc{ws.r[1], (long long)L * w, (long long)w}, xd, B, L, w, ws.A,
                          ws.r, 0, 0, st);
            if (e != hipSuccess) return hip_fail(e, "pcr_sweep");
            e = timed(DEEPPCR_KCLASS_UPDATE, 12.0 * n, 2.0 * n, st,
                      [&] { return launch_update_reduce(Z, xd.base, n, ws.red, st); });
            if (e != hipSuccess) return hip_fail(e, "update_reduce");
        }
        if (rule.residual) continue;
        unsigned ms[3];
        DEEPPCR_HIP(read_measures(ws.red, hw, st, ms));
        const unsigned mx = ms[0], mz = ms[1];
        if (iters_out) *iters_out = k + 1;
        if (measure_out) *measure_out = bits_to_float(mx);
        if (mx >= 0x7f800000u || mz >= 0x7f800000u) return DEEPPCR_ENONFINITE;
        const float m = bits_to_float(mx), zmax = bits_to_float(mz);
        if (rule.tol > 0.f && m < rule.tol * (zmax > 1.f ? zmax : 1.f)) return DEEPPCR_OK;
    }
    return rule.tol > 0.f ? DEEPPCR_ENOCONV : DEEPPCR_OK;
}

int pcr_solve_run(const float* J, const float* r, float* x, int B, int L, int w, int transpose,
                  void* workspace, hipStream_t st);

}  // namespace

extern "C" {

size_t deeppcr_workspace_bytes(int op, int B, int L, int w) {
    if (op < DEEPPCR_OP_PCR || op > DEEPPCR_OP_BWD || !sizes_ok(B, L, w)) return 0;
    return layout(op, B, L, w).total;
}

const char* deeppcr_status_string(int status) {
    switch (status) {
        case DEEPPCR_OK: return "ok";
        case DEEPPCR_EINVAL: return "invalid argument";
        case DEEPPCR_ENOCONV: return "Newton did not reach the tolerance within max_iter";
        case DEEPPCR_ENONFINITE: return "non-finite value in the Newton iterate";
        case DEEPPCR_EHIP: return "HIP runtime error";
        case DEEPPCR_EWORKSPACE: return "workspace too small";
        default: return "unknown status";
    }
}

const char* deeppcr_last_error(void) { return g_last_error; }

int pcr_solve_block_bidiag(const float* J, const float* r, float* x, int B, int L, int w,
                           int transpose, void* workspace, size_t workspace_bytes,
                           void* stream) {
    const SpanGuard span_guard;
    if (!J || !r || !x || !workspace || !sizes_ok(B, L, w) || (transpose != 0 && transpose != 1))
        return DEEPPCR_EINVAL;
    if (!aligned({J, r, x, workspace})) return DEEPPCR_EINVAL;
    const Layout lo = layout(DEEPPCR_OP_PCR, B, L, w);
    if (workspace_bytes < lo.total) return DEEPPCR_EWORKSPACE;
    const size_t nJ = (size_t)B * L * w * w * 4, nv = (size_t)B * L * w * 4;
    if (overlaps(x, nv, J, nJ) || overlaps(workspace, lo.total, J, nJ) ||
        overlaps(workspace, lo.total, r, nv) || overlaps(workspace, lo.total, x, nv))
        return DEEPPCR_EINVAL;
    if ((x != r) && overlaps(x, nv, r, nv)) return DEEPPCR_EINVAL;
    return pcr_solve_run(J, r, x, B, L, w, transpose, workspace, (hipStream_t)stream);
}

}  // extern "C"

namespace {

// The solve behind pcr_solve_block_bidiag and its no-allocation variant,
// after validation: the workspace (or the library's scratch) is carved by
// the same layout.
int pcr_solve_run(const float* J, const float* r, float* x, int B, int L, int w, int transpose,
                  void* workspace, hipStream_t st) {
    const Layout lo = layout(DEEPPCR_OP_PCR, B, L, w);
    Ws ws = carve(workspace, lo);
    const long long bw2 = (long long)L * w * w, w2 = (long long)w * w;
    BlockSrc A0;
    VecSrc r0;
    VecDst xd;
    if (!transpose) {
        A0 = BlockSrc{J, bw2, w2, 0};
        r0 = VecSrc{r, (long long)L * w, w};
        xd = VecDst{x, (long long)L * w, w};
    } else {
        // Transposed system in reversed row order: row m = L-1-l has operator
        // J_{L-m}^T and right-hand side r_{L-1-m}.
        A0 = BlockSrc{J + (long long)L * w2, bw2, -w2, 1};
        r0 = VecSrc{r + (long long)(L - 1) * w, (long long)L * w, -(long long)w};
        xd = VecDst{x + (long long)(L - 1) * w, (long long)L * w, -(long long)w};
    }
    hipError_t e = pcr_sweep(A0, r0, xd, B, L, w, ws.A, ws.r, 0, 0, st);
    if (e != hipSuccess) return hip_fail(e, "pcr_solve_block_bidiag");
    return DEEPPCR_OK;
}

}  // namespace

// ------------------------------------------------------ row-chunked solve
namespace {

struct ChunkLayout {
    size_t A[2], r[2], xin, total;
};

ChunkLayout chunk_layout(int B, int L, int w, int G) {
    const size_t nA = (size_t)B * L * w * w * sizeof(float);
    const size_t nr = (size_t)B * L * w * sizeof(float);
    const int Lc = (L + G - 1) / G;
    const size_t nx = (size_t)B * chunk_count(L, Lc) * w * sizeof(float);
    ChunkLayout lo{};
    size_t off = 0;
    lo.A[0] = off; off += align_up(nA);
    lo.A[1] = off; off += align_up(nA);
    lo.r[0] = off; off += align_up(nr);
    lo.r[1] = off; off += align_up(nr);
    lo.xin = off; off += align_up(nx);
    lo.total = off;
    return lo;
}

}  // namespace

extern "C" {

size_t deeppcr_chunked_workspace_bytes(int B, int L, int w, int G) {
    if (!block_sizes_ok(B, L, w) || G < 1) return 0;
    return chunk_layout(B, L, w, G).total;
}

int pcr_solve_block_bidiag_chunked(const float* J, const float* r, float* x, int B, int L, int w,
                                   int transpose, int G, void* workspace,
                                   size_t workspace_bytes, void* stream) {
    const SpanGuard span_guard;
    if (!J || !r || !x || !workspace || !block_sizes_ok(B, L, w) || G < 1 ||
        (transpose != 0 && transpose != 1))
        return DEEPPCR_EINVAL;
    if (!aligned({J, r, x, workspace})) return DEEPPCR_EINVAL;
    const ChunkLayout lo = chunk_layout(B, L, w, G);
    if (workspace_bytes < lo.total) return DEEPPCR_EWORKSPACE;
    const size_t nJ = (size_t)B * L * w * w * 4, nv = (size_t)B * L * w * 4;
    if (overlaps(x, nv, J, nJ) || overlaps(workspace, lo.total, J, nJ) ||
        overlaps(workspace, lo.total, r, nv) || overlaps(workspace, lo.total, x, nv))
        return DEEPPCR_EINVAL;
    if ((x != r) && overlaps(x, nv, r, nv)) return DEEPPCR_EINVAL;

    hipStream_t st = (hipStream_t)stream;
    char* base = (char*)workspace;
    float* wsA[2] = {(float*)(base + lo.A[0]), (float*)(base + lo.A[1])};
    float* wsr[2] = {(float*)(base + lo.r[0]), (float*)(base + lo.r[1])};
    float* xin = (float*)(base + lo.xin);
    const long long bw2 = (long long)L * w * w, w2 = (long long)w * w;
    const int rev = transpose;
    BlockSrc Ain;
    VecSrc rin;
    VecDst xd;
    if (!transpose) {
        Ain = BlockSrc{J, bw2, w2, 0};
        rin = VecSrc{r, (long long)L * w, w};
        xd = VecDst{x, (long long)L * w, w};
    } else {
        // reversed row order: internal row m = L-1-l has operator J_{L-m}^T
        Ain = BlockSrc{J + (long long)L * w2, bw2, -w2, 1};
        rin = VecSrc{r + (long long)(L - 1) * w, (long long)L * w, -(long long)w};
        xd = VecDst{x + (long long)(L - 1) * w, (long long)L * w, -(long long)w};
    }
    const int Lc = (L + G - 1) / G;
    // levels s = 1, 2, ... while s < Lc (a chunk of one row still takes one,
    // copying, level, which moves its block into the operator buffer); where
    // the width allows, only the first Kc - 6 of the Kc levels (at least one),
    // and the chains of at most 64 rows they leave by substitution
    int Kc = 0;
    for (long long t = 1; t < Lc; t *= 2) ++Kc;
    const int k0 = Kc - 6 > 1 ? Kc - 6 : 1;
    const bool chains = chunk_chain_width(w) && k0 < Kc;
    const int klev = chains ? k0 : (Kc > 1 ? Kc : 1);
    int k = 0;
    for (int s = 1; k < klev; s *= 2, ++k) {
        double bytes, flops;
        chunk_level_work(B, L, w, Lc, rev, s, &bytes, &flops);
        float* Aout = wsA[k & 1];
        float* rout = wsr[k & 1];
        hipError_t e = timed(DEEPPCR_KCLASS_PCR_LEVEL, bytes, flops, st, [&] {
            return launch_chunk_level(Ain, rin, Aout, rout, B, L, w, Lc, rev, s, st);
        });
        if (e != hipSuccess) return hip_fail(e, "pcr_solve_block_bidiag_chunked");
        Ain = BlockSrc{Aout, bw2, w2, 0};
        rin = VecSrc{rout, (long long)L * w, w};
    }
    const float* P = wsA[(k - 1) & 1];
    const float* q = wsr[(k - 1) & 1];
    if (chains) {
        double bytes, flops;
        chunk_chain_work(B, L, w, Lc, rev, 1 << k, &bytes, &flops);
        hipError_t e = timed(DEEPPCR_KCLASS_PCR_TAIL, bytes, flops, st, [&] {
            return launch_chunk_chain(P, q, wsA[k & 1], wsr[k & 1], B, L, w, Lc, rev, 1 << k, st);
        });
        if (e != hipSuccess) return hip_fail(e, "pcr_solve_block_bidiag_chunked");
        P = wsA[k & 1];
        q = wsr[k & 1];
    }
    const int nch = chunk_count(L, Lc);
    hipError_t e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * B * nch * (w2 + 2.0 * w),
                         2.0 * B * nch * w2, st,
                         [&] { return launch_chunk_carry(P, q, xin, B, L, w, Lc, rev, st); });
    if (e != hipSuccess) return hip_fail(e, "pcr_solve_block_bidiag_chunked");
    const double apply_rows = (double)B * (L - (transpose ? L - (nch - 1) * Lc : Lc));
    e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * (apply_rows * w2 + 2.0 * B * L * w),
              2.0 * apply_rows * w2, st,
              [&] { return launch_chunk_apply(P, q, xin, xd, B, L, w, Lc, rev, st); });
    if (e != hipSuccess) return hip_fail(e, "pcr_solve_block_bidiag_chunked");
    return DEEPPCR_OK;
}

}  // extern "C"

// ------------------------------------------------- no-allocation variant
// The scratch of pcr_solve_block_bidiag_noalloc: a fixed device array in
// place of the caller's workspace.  Each GPU holds its own copy (allocated
// when the library's code object is loaded on that GPU, kept until the
// process ends).  In host code `scratch` names a host-side stand-in, not
// the device array: host code uses only the address from
// hipGetSymbolAddress, kept per device.
static __device__ __align__(256) unsigned char scratch[DEEPPCR_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr size_t kScratchBytes = (size_t)DEEPPCR_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's scratch, looked up once per
// device (with that device current) and cached.
hipError_t scratch_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {

int pcr_solve_block_bidiag_noalloc(const float* J, const float* r, float* x, int B, int L,
                                   int w, int transpose, void* stream) {
    const SpanGuard span_guard;
    if (!J || !r || !x || !sizes_ok(B, L, w) || (transpose != 0 && transpose != 1))
        return DEEPPCR_EINVAL;
    if (!aligned({J, r, x})) return DEEPPCR_EINVAL;
    const size_t nJ = (size_t)B * L * w * w * 4, nv = (size_t)B * L * w * 4;
    if (overlaps(x, nv, J, nJ)) return DEEPPCR_EINVAL;
    if ((x != r) && overlaps(x, nv, r, nv)) return DEEPPCR_EINVAL;
    if (layout(DEEPPCR_OP_PCR, B, L, w).total > kScratchBytes) return DEEPPCR_EWORKSPACE;
    // no event is created or recorded during this call, whatever the
    // instrumentation setting
    const bool prof_on = g_prof.on;
    g_prof.on = false;
    void* ws = nullptr;
    hipError_t e = scratch_address(&ws);
    int status = e != hipSuccess ? hip_fail(e, "hipGetSymbolAddress(scratch)")
                                 : pcr_solve_run(J, r, x, B, L, w, transpose, ws,
                                                 (hipStream_t)stream);
    g_prof.on = prof_on;
    return status;
}

size_t deeppcr_noalloc_scratch_bytes(void) { return kScratchBytes; }

int deeppcr_newton_step(const float* J, const float* F, float* Z, int B, int L, int w, float tol,
                        void* workspace, size_t workspace_bytes, float* residual_out,
                        float* max_update_out, float* max_abs_out, void* stream) {
    const SpanGuard span_guard;
    if (!J || !F || !Z || !workspace || !sizes_ok(B, L, w)) return DEEPPCR_EINVAL;
    if (!(tol >= 0.f) || !std::isfinite(tol)) return DEEPPCR_EINVAL;
    if (!aligned({J, F, Z, workspace})) return DEEPPCR_EINVAL;
    const Layout lo = layout(DEEPPCR_OP_PCR, B, L, w);
    if (workspace_bytes < lo.total) return DEEPPCR_EWORKSPACE;
    const size_t nJ = (size_t)B * L * w * w * 4, nv = (size_t)B * L * w * 4;
    if (overlaps(Z, nv, J, nJ) || overlaps(Z, nv, F, nv) || overlaps(workspace, lo.total, J, nJ) ||
        overlaps(workspace, lo.total, F, nv) || overlaps(workspace, lo.total, Z, nv))
        return DEEPPCR_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    Ws ws = carve(workspace, lo);
    unsigned* hw = host_words();
    if (!hw) return hip_fail(hipErrorOutOfMemory, "hipHostMalloc");
    const long long n = (long long)B * L * w;
    // all reduction slots cleared, then r = F - Z with max |r|
    hipError_t e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * kRedWords, 0.0, st,
                         [&] { return launch_zero_words(ws.red, kRedWords, st); });
    if (e != hipSuccess) return hip_fail(e, "zero_words");
    e = timed(DEEPPCR_KCLASS_LAYER, 12.0 * n, (double)n, st,
              [&] { return launch_residual(F, Z, ws.r[1], n, ws.red, st); });
    if (e != hipSuccess) return hip_fail(e, "residual");
    // Eq. 3 with the caller's blocks (J[:, 0] unused) by PCR, then Z += dZ:
    // applied by the substitution pass of the last levels where the sweep
    // ends in one, else by the update kernel
    const BlockSrc J0{J, (long long)L * w * w, (long long)w * w, 0};
    const VecSrc r0{ws.r[1], (long long)L * w, (long long)w};
    if (tail_levels(B, L, w, 0) > 0) {
        e = pcr_sweep(J0, r0, VecDst{Z, (long long)L * w, (long long)w}, B, L, w, ws.A, ws.r, 0,
                      0, st, nullptr, ws.red);
        if (e != hipSuccess) return hip_fail(e, "pcr_sweep");
    } else {
        const VecDst xd{ws.r[(num_passes(B, L, w) + 1) & 1], (long long)L * w, (long long)w};
        e = pcr_sweep(J0, r0, xd, B, L, w, ws.A, ws.r, 0, 0, st);
        if (e != hipSuccess) return hip_fail(e, "pcr_sweep");
        e = timed(DEEPPCR_KCLASS_UPDATE, 12.0 * n, 2.0 * n, st,
                  [&] { return launch_update_reduce(Z, xd.base, n, ws.red, st); });
        if (e != hipSuccess) return hip_fail(e, "update_reduce");
    }
    unsigned ms[3];
    DEEPPCR_HIP(read_measures(ws.red, hw, st, ms));
    const unsigned mr = ms[2], mx = ms[0], mz = ms[1];
    if (residual_out) *residual_out = bits_to_float(mr);
    if (max_update_out) *max_update_out = bits_to_float(mx);
    if (max_abs_out) *max_abs_out = bits_to_float(mz);
    if (mr >= 0x7f800000u || mx >= 0x7f800000u || mz >= 0x7f800000u) return DEEPPCR_ENONFINITE;
    // the stopping test of the forward entry point, on this step's update
    const float m = bits_to_float(mx), zmax = bits_to_float(mz);
    if (tol > 0.f && m < tol * (zmax > 1.f ? zmax : 1.f)) return DEEPPCR_OK;
    return DEEPPCR_ENOCONV;
}

int deeppcr_mlp_forward(const float* W, const float* bias, const float* z0, float* Z, int B,
                        int L, int w, int layer, float alpha, float tol, int max_iter,
                        const float* Z_init, void* workspace, size_t workspace_bytes,
                        int* iters_out, float* last_update_out, void* stream) {
    const SpanGuard span_guard;
    const int c = check_forward_args(W, bias, z0, Z, Z_init, workspace, workspace_bytes, B, L, w,
                                     layer, alpha);
    if (c != DEEPPCR_OK) return c;
    if (!(tol >= 0.f) || !std::isfinite(tol) || max_iter < 1) return DEEPPCR_EINVAL;
    const StopRule rule{0, tol, 0.f, 0.f, max_iter};
    return newton_forward(W, bias, z0, Z, B, L, w, layer, alpha, rule, Z_init, workspace,
                          iters_out, last_update_out, (hipStream_t)stream);
}

int deeppcr_mlp_forward_residual(const float* W, const float* bias, const float* z0, float* Z,
                                 int B, int L, int w, int layer, float alpha, float atol,
                                 float rtol, int max_iter, const float* Z_init, void* workspace,
                                 size_t workspace_bytes, int* iters_out, float* residual_out,
                                 void* stream) {
    const SpanGuard span_guard;
    const int c = check_forward_args(W, bias, z0, Z, Z_init, workspace, workspace_bytes, B, L, w,
                                     layer, alpha);
    if (c != DEEPPCR_OK) return c;
    if (!(atol >= 0.f) || !std::isfinite(atol) || !(rtol >= 0.f) || !std::isfinite(rtol) ||
        max_iter < 0)
        return DEEPPCR_EINVAL;
    const StopRule rule{1, 0.f, atol, rtol, max_iter};
    return newton_forward(W, bias, z0, Z, B, L, w, layer, alpha, rule, Z_init, workspace,
                          iters_out, residual_out, (hipStream_t)stream);
}

int deeppcr_mlp_backward(const float* W, const float* bias, const float* z0, const float* Z,
                         const float* G, float* Lambda, float* dz0, float* dW, float* db, int B,
                         int L, int w, int layer, float alpha, void* workspace,
                         size_t workspace_bytes, void* stream) {
    const SpanGuard span_guard;
    if (!W || !bias || !z0 || !Z || !G || !Lambda || !dz0 || !dW || !db || !workspace ||
        !sizes_ok(B, L, w))
        return DEEPPCR_EINVAL;
    if (layer < 0 || layer >= kNumLayerKinds) return DEEPPCR_EINVAL;
    if (!std::isfinite(alpha)) return DEEPPCR_EINVAL;
    if (!aligned({W, bias, z0, Z, G, Lambda, dz0, dW, db, workspace})) return DEEPPCR_EINVAL;
    const Layout lo = layout(DEEPPCR_OP_BWD, B, L, w);
    if (workspace_bytes < lo.total) return DEEPPCR_EWORKSPACE;
    const size_t nv = (size_t)B * L * w * 4, nW = (size_t)L * w * w * 4;
    const void* ins[] = {W, bias, z0, Z, G};
    const size_t nins[] = {nW, (size_t)L * w * 4, (size_t)B * w * 4, nv, (size_t)B * w * 4};
    void* outs[] = {Lambda, dz0, dW, db};
    const size_t nouts[] = {nv, (size_t)B * w * 4, nW, (size_t)L * w * 4};
    for (int i = 0; i < 4; ++i) {
        if (overlaps(workspace, lo.total, outs[i], nouts[i])) return DEEPPCR_EINVAL;
        for (int j = 0; j < 5; ++j)
            if (overlaps(outs[i], nouts[i], ins[j], nins[j])) return DEEPPCR_EINVAL;
        for (int j = i + 1; j < 4; ++j)
            if (overlaps(outs[i], nouts[i], outs[j], nouts[j])) return DEEPPCR_EINVAL;
    }
    for (int j = 0; j < 5; ++j)
        if (overlaps(workspace, lo.total, ins[j], nins[j])) return DEEPPCR_EINVAL;

    hipStream_t st = (hipStream_t)stream;
    Ws ws = carve(workspace, lo);
    const double w2 = (double)w * w;
    // w = 32, 64, 128 with paired levels: the first PCR pass forms the blocks
    // from the weights and c d, so the assembly writes only c d and the
    // right-hand side
    const bool from_weights = first_level_count(B, L, w) == 2;
    const BwdArgs bw{W, ws.dscale, layer_residual(layer) ? 1 : 0};
    const double jbytes = from_weights ? 0.0 : 4.0 * B * L * w2;
    hipError_t e = timed(DEEPPCR_KCLASS_LAYER, jbytes + 4.0 * B * L * 3.0 * w,
                         (double)B * L * (from_weights ? 2.0 : 3.0) * w2, st, [&] {
        return launch_backward_assemble(W, bias, z0, Z, G, from_weights ? nullptr : ws.A[1],
                                        ws.r[1], ws.dscale, B, L, w, layer, alpha, st);
    });
    if (e != hipSuccess) return hip_fail(e, "backward_assemble");
    const VecDst lam{Lambda + (long long)(L - 1) * w, (long long)L * w, -(long long)w};
    e = pcr_sweep(BlockSrc{ws.A[1], (long long)L * w * w, (long long)w * w,
                           backward_blocks_transposed(w) ? 1 : 0},
                  VecSrc{ws.r[1], (long long)L * w, (long long)w}, lam, B, L, w, ws.A, ws.r, 0, 0,
                  st, from_weights ? &bw : nullptr);
    if (e != hipSuccess) return hip_fail(e, "pcr_sweep");
    e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * (w2 + 3.0 * B * w), 2.0 * B * w2, st, [&] {
        return launch_dz0(W, ws.dscale, Lambda, dz0, B, L, w, layer, st);
    });
    if (e != hipSuccess) return hip_fail(e, "dz0");
    e = timed(DEEPPCR_KCLASS_WGRAD, 4.0 * (3.0 * B * L * w + L * (w2 + w)), 2.0 * B * L * w2, st,
              [&] { return launch_wgrad(z0, Z, ws.dscale, Lambda, dW, db, B, L, w, st); });
    if (e != hipSuccess) return hip_fail(e, "wgrad");
    return DEEPPCR_OK;
}

size_t deeppcr_resnet_workspace_bytes(int op, int B, int L, int w, int skip) {
    if ((op != DEEPPCR_OP_FWD && op != DEEPPCR_OP_BWD) || !resnet_shape_ok(B, L, w, skip, 0))
        return 0;
    return resnet_layout(op, B, L / skip, w).total;
}

int deeppcr_resnet_forward(const float* W, const float* bias, const float* z0, float* Z, int B,
                           int L, int w, int skip, int act, float tol, int max_iter,
                           const float* Z_init, void* workspace, size_t workspace_bytes,
                           int* iters_out, float* last_update_out, void* stream) {
    const SpanGuard span_guard;
    if (!W || !bias || !z0 || !Z || !workspace || !resnet_shape_ok(B, L, w, skip, act))
        return DEEPPCR_EINVAL;
    if (!(tol >= 0.f) || !std::isfinite(tol) || max_iter < 1) return DEEPPCR_EINVAL;
    if (!aligned({W, bias, z0, Z, Z_init, workspace})) return DEEPPCR_EINVAL;
    const int G = L / skip;
    const Layout lo = resnet_layout(DEEPPCR_OP_FWD, B, G, w);
    if (workspace_bytes < lo.total) return DEEPPCR_EWORKSPACE;
    const size_t nv = (size_t)B * L * w * 4;
    if (overlaps(workspace, lo.total, Z, nv) ||
        overlaps(workspace, lo.total, W, (size_t)L * w * w * 4) ||
        overlaps(workspace, lo.total, z0, (size_t)B * w * 4) ||
        overlaps(workspace, lo.total, bias, (size_t)L * w * 4) ||
        overlaps(workspace, lo.total, Z_init, Z_init ? nv : 0))
        return DEEPPCR_EINVAL;
    if (Z_init && Z_init != Z && overlaps(Z_init, nv, Z, nv)) return DEEPPCR_EINVAL;

    hipStream_t st = (hipStream_t)stream;
    Ws ws = carve(workspace, lo);
    float* X = (float*)((char*)workspace + lo.dscale);
    unsigned* hw = host_words();
    if (!hw) return hip_fail(hipErrorOutOfMemory, "hipHostMalloc");
    if (iters_out) *iters_out = 0;
    if (last_update_out) *last_update_out = 0.f;
    const long long n = (long long)B * G * w;
    const double w2 = (double)w * w;
    if (Z_init) {
        // X^0[b, g] = Z_init[b, g*skip + skip - 1]
        const VecSrc src{Z_init + (long long)(skip - 1) * w, (long long)L * w, (long long)skip * w};
        const VecDst dst{X, (long long)G * w, (long long)w};
        hipError_t e = timed(DEEPPCR_KCLASS_OTHER, 8.0 * n, 0.0, st,
                             [&] { return launch_copy_rows(src, dst, B, G, w, st); });
        if (e != hipSuccess) return hip_fail(e, "copy_rows");
    } else {
        hipError_t e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * n, 2.0 * B * skip * w2, st, [&] {
            return launch_resnet_initial_guess(W, bias, z0, X, B, G, w, skip, act, st);
        });
        if (e != hipSuccess) return hip_fail(e, "resnet_initial_guess");
    }
    const VecDst xd{ws.r[(num_passes(B, G, w) + 1) & 1], (long long)G * w, (long long)w};
    // block evaluation: W once, X read twice, blocks and residuals written;
    // flops: the s - 1 block products and the s mat-vecs per block
    const double eval_bytes = 4.0 * ((double)L * w2 + (double)B * G * (w2 + 3.0 * w));
    const double eval_flops = (double)B * G * ((skip - 1) * 2.0 * w2 * w + skip * 2.0 * w2);
    int status = tol > 0.f ? DEEPPCR_ENOCONV : DEEPPCR_OK;
    const bool upd_in_tail = tail_levels(B, G, w, 0) > 0;
    for (int k = 1; k <= max_iter; ++k) {
        hipError_t e = timed(DEEPPCR_KCLASS_LAYER, eval_bytes, eval_flops, st, [&] {
            return launch_resnet_block_eval(W, bias, z0, X, ws.A[1], ws.r[1], ws.red, B, G, w,
                                            skip, act, st);
        });
        if (e != hipSuccess) return hip_fail(e, "resnet_block_eval");
        if (upd_in_tail) {
            // the substitution pass of the last levels adds the solution to
            // the iterate and reduces the convergence maxima itself (the
            // block evaluation cleared their slots)
            e = pcr_sweep(BlockSrc{ws.A[1], (long long)G * w * w, (long long)w * w, 0},
                          VecSrc{ws.r[1], (long long)G * w, (long long)w},
                          VecDst{X, (long long)G * w, (long long)w}, B, G, w, ws.A, ws.r, 0, 0,
                          st, nullptr, ws.red);
            if (e != hipSuccess) return hip_fail(e, "pcr_sweep");
        } else {
            e = pcr_sweep(BlockSrc{ws.A[1], (long long)G * w * w, (long long)w * w, 0},
                          VecSrc{ws.r[1], (long long)G * w, (long long)w}, xd, B, G, w, ws.A,
                          ws.r, 0, 0, st);
            if (e != hipSuccess) return hip_fail(e, "pcr_sweep");
            e = timed(DEEPPCR_KCLASS_UPDATE, 12.0 * n, 2.0 * n, st,
                      [&] { return launch_update_reduce(X, xd.base, n, ws.red, st); });
            if (e != hipSuccess) return hip_fail(e, "update_reduce");
        }
        unsigned ms[3];
        DEEPPCR_HIP(read_measures(ws.red, hw, st, ms));
        const unsigned mx = ms[0], mz = ms[1];
        if (iters_out) *iters_out = k;
        if (last_update_out) *last_update_out = bits_to_float(mx);
        if (mx >= 0x7f800000u || mz >= 0x7f800000u) {
            status = DEEPPCR_ENONFINITE;
            break;
        }
        const float m = bits_to_float(mx), zmax = bits_to_float(mz);
        if (tol > 0.f && m < tol * (zmax > 1.f ? zmax : 1.f)) {
            status = DEEPPCR_OK;
            break;
        }
    }
    // every layer output from the block outputs
    hipError_t e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * ((double)L * w2 + 2.0 * B * L * w),
                         2.0 * B * (L - G) * w2, st, [&] {
                             return launch_resnet_expand(W, bias, z0, X, Z, B, G, w, skip, act,
                                                         st);
                         });
    if (e != hipSuccess) return hip_fail(e, "resnet_expand");
    return status;
}

int deeppcr_resnet_backward(const float* W, const float* z0, const float* Z, const float* G_,
                            float* Lambda, float* dz0, float* dW, float* db, int B, int L, int w,
                            int skip, int act, void* workspace, size_t workspace_bytes,
                            void* stream) {
    const SpanGuard span_guard;
    if (!W || !z0 || !Z || !G_ || !Lambda || !dz0 || !dW || !db || !workspace ||
        !resnet_shape_ok(B, L, w, skip, act))
        return DEEPPCR_EINVAL;
    if (!aligned({W, z0, Z, G_, Lambda, dz0, dW, db, workspace})) return DEEPPCR_EINVAL;
    const int G = L / skip;
    const Layout lo = resnet_layout(DEEPPCR_OP_BWD, B, G, w);
    if (workspace_bytes < lo.total) return DEEPPCR_EWORKSPACE;
    const size_t nv = (size_t)B * L * w * 4, nW = (size_t)L * w * w * 4;
    const void* ins[] = {W, z0, Z, G_};
    const size_t nins[] = {nW, (size_t)B * w * 4, nv, (size_t)B * w * 4};
    void* outs[] = {Lambda, dz0, dW, db};
    const size_t nouts[] = {nv, (size_t)B * w * 4, nW, (size_t)L * w * 4};
    for (int i = 0; i < 4; ++i) {
        if (overlaps(workspace, lo.total, outs[i], nouts[i])) return DEEPPCR_EINVAL;
        if (overlaps(workspace, lo.total, ins[i], nins[i])) return DEEPPCR_EINVAL;
        for (int j = 0; j < 4; ++j)
            if (overlaps(outs[i], nouts[i], ins[j], nins[j])) return DEEPPCR_EINVAL;
        for (int j = i + 1; j < 4; ++j)
            if (overlaps(outs[i], nouts[i], outs[j], nouts[j])) return DEEPPCR_EINVAL;
    }
    hipStream_t st = (hipStream_t)stream;
    Ws ws = carve(workspace, lo);
    const double w2 = (double)w * w;
    // blocks of the transposed block system (reversed rows) and its right-hand side
    hipError_t e = timed(DEEPPCR_KCLASS_LAYER,
                         4.0 * ((double)L * w2 + (double)B * L * w + (double)B * G * (w2 + w)),
                         (double)B * G * (skip - 1) * 2.0 * w2 * w, st, [&] {
                             return launch_resnet_block_jac(W, z0, Z, G_, ws.A[1], ws.r[1], B, G,
                                                            w, skip, act, st);
                         });
    if (e != hipSuccess) return hip_fail(e, "resnet_block_jac");
    // block-output adjoints mu (natural order) from the transposed solve
    float* mu = ws.r[(num_passes(B, G, w) + 1) & 1];
    const VecDst xd{mu + (long long)(G - 1) * w, (long long)G * w, -(long long)w};
    e = pcr_sweep(BlockSrc{ws.A[1], (long long)G * w * w, (long long)w * w, 1},
                  VecSrc{ws.r[1], (long long)G * w, (long long)w}, xd, B, G, w, ws.A, ws.r, 0, 0,
                  st);
    if (e != hipSuccess) return hip_fail(e, "pcr_sweep");
    e = timed(DEEPPCR_KCLASS_OTHER, 4.0 * ((double)L * w2 + 2.0 * B * L * w),
              2.0 * B * L * w2, st, [&] {
                  return launch_resnet_intra_adjoint(W, z0, Z, mu, Lambda, dz0, B, G, w, skip,
                                                     act, st);
              });
    if (e != hipSuccess) return hip_fail(e, "resnet_intra_adjoint");
    e = timed(DEEPPCR_KCLASS_WGRAD, 4.0 * (2.0 * B * L * w + L * (w2 + w)), 2.0 * B * L * w2, st,
              [&] { return launch_wgrad_pre(z0, Z, Lambda, dW, db, B, L, w, act, st); });
    if (e != hipSuccess) return hip_fail(e, "wgrad");
    return DEEPPCR_OK;
}

int deeppcr_resnet_seq_forward(const float* W, const float* bias, const float* z0, float* Z,
                               int B, int L, int w, int skip, int act, int launch_per_layer,
                               void* stream) {
    const SpanGuard span_guard;
    if (!W || !bias || !z0 || !Z || !resnet_shape_ok(B, L, w, skip, act) ||
        (launch_per_layer != 0 && launch_per_layer != 1))
        return DEEPPCR_EINVAL;
    if (!aligned({W, bias, z0, Z})) return DEEPPCR_EINVAL;
    const size_t nv = (size_t)B * L * w * 4;
    if (overlaps(Z, nv, W, (size_t)L * w * w * 4) || overlaps(Z, nv, bias, (size_t)L * w * 4) ||
        overlaps(Z, nv, z0, (size_t)B * w * 4))
        return DEEPPCR_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    const int step = launch_per_layer ? 1 : L;
    for (int l0 = 0; l0 < L; l0 += step) {
        const int l1 = l0 + step;
        const double n = (double)(l1 - l0);
        hipError_t e = timed(DEEPPCR_KCLASS_SEQUENTIAL, 4.0 * n * ((double)w * w + 2.0 * B * w),
                             2.0 * B * n * w * w, st, [&] {
                                 return launch_resnet_seq_forward(W, bias, z0, Z, B, L, w, skip,
                                                                  act, l0, l1, st);
                             });
        if (e != hipSuccess) return hip_fail(e, "resnet_seq_forward");
    }
    return DEEPPCR_OK;
}

int deeppcr_resnet_seq_backward(const float* W, const float* z0, const float* Z, const float* G,
                                float* Lambda, float* dz0, int B, int L, int w, int skip, int act,
                                int launch_per_layer, void* stream) {
    const SpanGuard span_guard;
    if (!W || !z0 || !Z || !G || !Lambda || !dz0 || !resnet_shape_ok(B, L, w, skip, act) ||
        (launch_per_layer != 0 && launch_per_layer != 1))
        return DEEPPCR_EINVAL;
    if (!aligned({W, z0, Z, G, Lambda, dz0})) return DEEPPCR_EINVAL;
    const size_t nv = (size_t)B * L * w * 4, nb = (size_t)B * w * 4;
    const void* ins[] = {W, z0, Z, G};
    const size_t nins[] = {(size_t)L * w * w * 4, nb, nv, nb};
    for (int j = 0; j < 4; ++j)
        if (overlaps(Lambda, nv, ins[j], nins[j]) || overlaps(dz0, nb, ins[j], nins[j]))
            return DEEPPCR_EINVAL;
    if (overlaps(Lambda, nv, dz0, nb)) return DEEPPCR_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    const int step = launch_per_layer ? 1 : L;
    for (int l1 = L; l1 > 0; l1 -= step) {
        const int l0 = l1 - step;
        const double n = (double)(l1 - l0);
        hipError_t e = timed(DEEPPCR_KCLASS_SEQUENTIAL, 4.0 * n * ((double)w * w + 3.0 * B * w),
                             2.0 * B * n * w * w, st, [&] {
                                 return launch_resnet_seq_backward(W, z0, Z, G, Lambda, dz0, B, L,
                                                                   w, skip, act, l0, l1, st);
                             });
        if (e != hipSuccess) return hip_fail(e, "resnet_seq_backward");
    }
    return DEEPPCR_OK;
}

int deeppcr_seq_forward(const float* W, const float* bias, const float* z0, float* Z, int B,
                        int L, int w, int layer, float alpha, int launch_per_layer, void* stream) {
    const SpanGuard span_guard;
    if (!W || !bias || !z0 || !Z || !sizes_ok(B, L, w)) return DEEPPCR_EINVAL;
    if (layer < 0 || layer >= kNumLayerKinds || !std::isfinite(alpha)) return DEEPPCR_EINVAL;
    if (launch_per_layer != 0 && launch_per_layer != 1) return DEEPPCR_EINVAL;
    if (!aligned({W, bias, z0, Z})) return DEEPPCR_EINVAL;
    const size_t nv = (size_t)B * L * w * 4;
    if (overlaps(Z, nv, W, (size_t)L * w * w * 4) || overlaps(Z, nv, bias, (size_t)L * w * 4) ||
        overlaps(Z, nv, z0, (size_t)B * w * 4))
        return DEEPPCR_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    if (wide_width(w)) {
        // one launch per layer whatever launch_per_layer says: a layer's
        // matrix is spread over the chip (one workgroup per system cannot
        // stream a block this size at speed)
        for (int l = 0; l < L; ++l) {
            hipError_t e = timed(DEEPPCR_KCLASS_SEQUENTIAL, 4.0 * ((double)w * w + 2.0 * B * w),
                                 2.0 * B * w * w, st, [&] {
                return launch_seq_forward_wide(W, bias, z0, Z, B, L, w, layer, alpha, l, st);
            });
            if (e != hipSuccess) return hip_fail(e, "seq_forward");
        }
        return DEEPPCR_OK;
    }
    const int step = launch_per_layer ? 1 : L;
    for (int l0 = 0; l0 < L; l0 += step) {
        const int l1 = l0 + step < L ? l0 + step : L;
        const double n = l1 - l0;
        hipError_t e = timed(DEEPPCR_KCLASS_SEQUENTIAL, 4.0 * n * ((double)w * w + 2.0 * B * w),
                             2.0 * n * B * w * w, st, [&] {
            return launch_seq_forward(W, bias, z0, Z, B, L, w, layer, alpha, l0, l1, st);
        });
        if (e != hipSuccess) return hip_fail(e, "seq_forward");
    }
    return DEEPPCR_OK;
}

int deeppcr_seq_backward(const float* W, const float* bias, const float* z0, const float* Z,
                         const float* G, float* Lambda, float* dz0, int B, int L, int w, int layer,
                         float alpha, int launch_per_layer, void* stream) {
    const SpanGuard span_guard;
    if (!W || !bias || !z0 || !Z || !G || !Lambda || !dz0 || !sizes_ok(B, L, w)) return DEEPPCR_EINVAL;
    if (layer < 0 || layer >= kNumLayerKinds || !std::isfinite(alpha)) return DEEPPCR_EINVAL;
    if (launch_per_layer != 0 && launch_per_layer != 1) return DEEPPCR_EINVAL;
    if (!aligned({W, bias, z0, Z, G, Lambda, dz0})) return DEEPPCR_EINVAL;
    const size_t nv = (size_t)B * L * w * 4, nb = (size_t)B * w * 4;
    const void* ins[] = {W, bias, z0, Z, G};
    const size_t nins[] = {(size_t)L * w * w * 4, (size_t)L * w * 4, nb, nv, nb};
    for (int j = 0; j < 5; ++j)
        if (overlaps(Lambda, nv, ins[j], nins[j]) || overlaps(dz0, nb, ins[j], nins[j]))
            return DEEPPCR_EINVAL;
    if (overlaps(Lambda, nv, dz0, nb)) return DEEPPCR_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    if (wide_width(w)) {
        // per layer (see deeppcr_seq_forward): the scaled adjoint, then its
        // product with W_l^T
        for (int l = L - 1; l >= 0; --l) {
            hipError_t e = timed(DEEPPCR_KCLASS_SEQUENTIAL, 4.0 * (2.0 * w * w + 4.0 * B * w),
                                 4.0 * B * w * w, st, [&] {
                return launch_seq_backward_wide(W, bias, z0, Z, G, Lambda, dz0, B, L, w, layer,
                                                alpha, l, st);
            });
            if (e != hipSuccess) return hip_fail(e, "seq_backward");
        }
        return DEEPPCR_OK;
    }
    const int step = launch_per_layer ? 1 : L;
    for (int l1 = L; l1 > 0; l1 -= step) {
        const int l0 = l1 - step > 0 ? l1 - step : 0;
        const double n = l1 - l0;
        hipError_t e = timed(DEEPPCR_KCLASS_SEQUENTIAL, 4.0 * n * ((double)w * w + 3.0 * B * w),
                             4.0 * n * B * w * w, st, [&] {
            return launch_seq_backward(W, bias, z0, Z, G, Lambda, dz0, B, L, w, layer, alpha, l0,
                                       l1, st);
        });
        if (e != hipSuccess) return hip_fail(e, "seq_backward");
    }
    return DEEPPCR_OK;
}

void deeppcr_release_thread_state(void) {
    (void)prof_break();
    for (auto& p : g_prof.pending) {
        (void)hipEventSynchronize(p.e1);
        if (!p.share0) (void)hipEventDestroy(p.e0);
        (void)hipEventDestroy(p.e1);
    }
    g_prof.pending.clear();
    for (hipEvent_t e : g_prof.pool) (void)hipEventDestroy(e);
    g_prof.pool.clear();
    if (g_host_words) {
        (void)hipHostFree(g_host_words);
        g_host_words = nullptr;
    }
}

int deeppcr_profile_enable(int on) {
    (void)prof_break();
    g_prof.on = on != 0;
    return DEEPPCR_OK;
}

int deeppcr_profile_select(unsigned class_mask) {
    (void)prof_break();
    g_prof.mask = class_mask;
    return DEEPPCR_OK;
}

void deeppcr_profile_reset(void) {
    (void)prof_break();
    for (auto& p : g_prof.pending) {
        (void)hipEventSynchronize(p.e1);
        if (!p.share0) g_prof.pool.push_back(p.e0);
        g_prof.pool.push_back(p.e1);
    }
    g_prof.pending.clear();
    for (int c = 0; c < DEEPPCR_KCLASS_COUNT; ++c) {
        g_prof.launches[c] = 0;
        g_prof.ms[c] = g_prof.bytes[c] = g_prof.flops[c] = 0.0;
    }
}

int deeppcr_profile_read(int kclass, long long* launches, double* total_ms, double* alg_bytes,
                         double* alg_flops) {
    if (kclass < 0 || kclass >= DEEPPCR_KCLASS_COUNT) return DEEPPCR_EINVAL;
    {
        hipError_t e = prof_break();
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
    }
    for (auto& p : g_prof.pending) {
        hipError_t e = hipEventSynchronize(p.e1);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, p.e0, p.e1);
        if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
        g_prof.launches[p.kclass] += p.n;
        g_prof.ms[p.kclass] += ms;
        g_prof.bytes[p.kclass] += p.bytes;
        g_prof.flops[p.kclass] += p.flops;
        if (!p.share0) g_prof.pool.push_back(p.e0);
        g_prof.pool.push_back(p.e1);
    }
    g_prof.pending.clear();
    if (launches) *launches = g_prof.launches[kclass];
    if (total_ms) *total_ms = g_prof.ms[kclass];
    if (alg_bytes) *alg_bytes = g_prof.bytes[kclass];
    if (alg_flops) *alg_flops = g_prof.flops[kclass];
    return DEEPPCR_OK;
}

}  // extern "C"
