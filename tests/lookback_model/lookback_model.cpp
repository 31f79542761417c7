// lookback_model.cpp -- a CPU model of the single-pass scans' cross-tile
// protocol, for randomised interleavings under ThreadSanitizer.
//
// TEST INFRASTRUCTURE.  The GPU dispatcher runs workgroups in one natural
// order; this model runs the same state machine with worker threads that
// take workgroups in dispatch order and are delayed at random points, so
// publication orders the hardware rarely produces occur here.  It models:
//
//   diagonal forward scan (memoroid_scan_diag): per-chain wrapping ticket
//   counters (two calls per cycle) giving the tile's place and the call's
//   epoch parity -- or, as the FFM forward keeps them, one counter per
//   (chain, group of G workgroups), the n-th ticket of counter (chain, x)
//   being position G n + x, with the grid padded to whole groups; two banks of self-validating descriptor words (all ones =
//   unpublished, NaN canonicalised); the tile publishing its aggregate, or
//   its inclusive prefix when it holds a begin step; the idle bank's words
//   cleared by their owner for the next call; the look-back folding
//   aggregates until an inclusive word closes the walk; the begin-count
//   words of the episode index (own / inclusive counts); the workspace
//   signature (bound by the first call, poisoned by a call with another
//   layout, every tile of that call standing down);
//
//   discounted return (memoroid_discounted_return): tiles ordered by
//   workgroup index from the tape's end, one epoch word per tile, the same
//   two banks, and the fallback that computes an awaited tile's map from
//   its inputs after a number of polls without progress.
//
// The resettable operator is the Section 4 reset theorem's, applied to the
// diagonal monoid (a, x) . (a', x') = (a'a, a'x + x') and to the return's
// monoid (App. D), carried as selects.
//
// Input: a directory holding the problems (raw little-endian arrays written
// by the test from the seeded generators, with the fp64 oracle's results and
// magnitude companions).  Output: one line per check; exit status 0 when
// every expectation holds (for a mutation: when the model detects it).
//
//   lookback_model <dir> diag <schedules> <mutation>
//   lookback_model <dir> diag_grouped <schedules> <mutation>
//   lookback_model <dir> return <schedules> <mutation>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <functional>
#include <mutex>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <string>
#include <thread>
#include <vector>

namespace {

// ------------------------------------------------------------- mutations
// Each alters one step of the protocol; the test expects the model to catch
// every one (a wrong result, a missed stand-down, or a wait that gives up).
enum Mutation {
    kNone = 0,
    kNoIdleClear,        // tiles leave the idle bank's words as they are
    kOneBank,            // every call publishes into bank 0
    kWrapEveryCall,      // counters wrap every call (bound n - 1): epoch parity lost
    kNoSignature,        // tiles ignore the workspace signature
    kNoPoison,           // a call with a foreign signature stands down without poisoning
    kNoCanon,            // NaN published as is (an all-ones NaN reads as unpublished)
    kEpochNotStored,     // return tiles do not store their epoch word back
    kFallbackWrongTile,  // the fallback folds the map of the tile after the awaited one
    kCountOwnAsIncl,     // a tile's own begin count is published as inclusive
    kMutations
};

constexpr uint32_t kEmpty32 = 0xFFFFFFFFu;
constexpr uint64_t kEmpty64 = 0xFFFFFFFFFFFFFFFFull;
constexpr uint64_t kSigPoisoned = 0;
constexpr uint64_t kCountOwn = 1ull << 62, kCountIncl = 2ull << 62, kCountValue = kCountOwn - 1;
constexpr uint32_t kMaxPolls = 200000;

// relaxed atomic accesses of plain words (the kernels' agent-scope relaxed
// loads and stores); plain stores stay plain, so ThreadSanitizer reports any
// of them that races with a reader
template <class T> T peek(const T* p) { return __atomic_load_n(p, __ATOMIC_RELAXED); }
template <class T> void publish(T* p, T v) { __atomic_store_n(p, v, __ATOMIC_RELAXED); }

struct Rng {
    std::mt19937_64 g;
    explicit Rng(uint64_t s) : g(s) {}
    uint32_t below(uint32_t n) { return (uint32_t)(g() % n); }
};

// a random pause: nothing, a few yields, or (rarely) a short sleep
void jitter(Rng& r) {
    const uint32_t k = r.below(64);
    if (k < 40) return;
    if (k < 63) {
        for (uint32_t i = 0, n = 1 + r.below(4); i < n; ++i) std::this_thread::yield();
        return;
    }
    std::this_thread::sleep_for(std::chrono::microseconds(1 + r.below(20)));
}

uint32_t fbits(float f) { uint32_t u; std::memcpy(&u, &f, 4); return u; }
float bitsf(uint32_t u) { float f; std::memcpy(&f, &u, 4); return f; }
float canon(float v, int mut) { return (v != v && mut != kNoCanon) ? bitsf(0x7FC00000u) : v; }
uint64_t pack2(float lo, float hi, int mut) {
    return (uint64_t)fbits(canon(lo, mut)) | ((uint64_t)fbits(canon(hi, mut)) << 32);
}
float lo_of(uint64_t w) { return bitsf((uint32_t)w); }
float hi_of(uint64_t w) { return bitsf((uint32_t)(w >> 32)); }

template <class T>
bool read_file(const std::string& path, std::vector<T>& out, size_t n) {
    FILE* f = std::fopen(path.c_str(), "rb");
    if (!f) return false;
    out.resize(n);
    const size_t got = n ? std::fread(out.data(), sizeof(T), n, f) : 0;
    std::fclose(f);
    return got == n;
}

// A pool of worker threads standing in for the GPU's compute units.
// launch(n, fn) hands workgroups 0 .. n - 1 out in order; fn(g, rng) runs
// one workgroup; launch returns once all have finished (the kernel
// boundary, which orders one call's memory accesses before the next call's).
class Pool {
public:
    Pool(int workers, uint64_t seed) : seed_(seed) {
        for (int w = 0; w < workers; ++w) threads_.emplace_back([this, w] { loop(w); });
    }
    ~Pool() {
        {
            std::unique_lock<std::mutex> lk(mu_);
            quit_ = true;
        }
        cv_.notify_all();
        for (auto& t : threads_) t.join();
    }
    template <class F>
    void launch(int64_t n, F fn) {
        std::function<void(int64_t, Rng&)> f = fn;
        {
            std::unique_lock<std::mutex> lk(mu_);
            job_ = &f;
            n_ = n;
            next_.store(0, std::memory_order_relaxed);
            done_ = 0;
            ++gen_;
        }
        cv_.notify_all();
        std::unique_lock<std::mutex> lk(mu_);
        done_cv_.wait(lk, [&] { return done_ == (int)threads_.size(); });
        job_ = nullptr;
    }

private:
    void loop(int w) {
        Rng r(seed_ * 1000003ull + (uint64_t)w * 7919ull);
        uint64_t seen = 0;
        while (true) {
            std::function<void(int64_t, Rng&)>* job;
            int64_t n;
            {
                std::unique_lock<std::mutex> lk(mu_);
                cv_.wait(lk, [&] { return quit_ || gen_ != seen; });
                if (quit_) return;
                seen = gen_;
                job = job_;
                n = n_;
            }
            while (true) {
                const int64_t g = next_.fetch_add(1, std::memory_order_relaxed);
                if (g >= n) break;
                jitter(r);
                (*job)(g, r);
            }
            {
                std::unique_lock<std::mutex> lk(mu_);
                ++done_;
            }
            done_cv_.notify_all();
        }
    }
    uint64_t seed_;
    std::vector<std::thread> threads_;
    std::mutex mu_;
    std::condition_variable cv_, done_cv_;
    std::function<void(int64_t, Rng&)>* job_ = nullptr;
    int64_t n_ = 0;
    std::atomic<int64_t> next_{0};
    int done_ = 0;
    uint64_t gen_ = 0;
    bool quit_ = false;
};

// ------------------------------------------------------ diagonal forward scan
struct DiagProblem {
    int64_t B = 0, T = 0, d = 0;
    std::vector<float> a, x;          // [B][T][d]
    std::vector<uint8_t> start;       // [B][T]
    std::vector<double> ref, mag;     // oracle's h and magnitude companion
    std::vector<int32_t> idx;         // oracle's episode index
};

// Workspace of one layout (F features per chain, L steps per tile).
struct DiagWs {
    int64_t F = 0, L = 0, nt = 0, nfb = 0, nch = 0, ntiles = 0, B = 0;
    int64_t groups = 1;               // tile counters per chain (G)
    uint64_t sig = kEmpty64;          // header: signature word
    uint32_t timeout = kEmpty32;      // header: a wait gave up
    std::vector<uint32_t> ctr;        // per-chain ticket counters
    std::vector<uint64_t> agg[2];     // [tile * nch + chain][F]
    std::vector<uint32_t> incl[2];
    std::vector<uint64_t> cnt[2];     // [tile][B] begin-count words
    void size_for(int64_t Bq, int64_t T, int64_t d, int64_t Fq, int64_t Lq) {
        B = Bq; F = Fq; L = Lq;
        nt = (T + L - 1) / L;
        nfb = (d + F - 1) / F;
        nch = B * nfb;
        ntiles = nt * nch;
        ctr.assign((size_t)(nch * groups), 0);
        for (int k = 0; k < 2; ++k) {
            agg[k].assign((size_t)(ntiles * F), 0);
            incl[k].assign((size_t)(ntiles * F), 0);
            cnt[k].assign((size_t)(nt * B), 0);
        }
    }
    void prepare() {       // memoroid_workspace_prepare: all-ones bytes
        sig = kEmpty64;
        timeout = kEmpty32;
        for (auto& c : ctr) c = kEmpty32;
        for (int k = 0; k < 2; ++k) {
            for (auto& w : agg[k]) w = kEmpty64;
            for (auto& w : incl[k]) w = kEmpty32;
            for (auto& w : cnt[k]) w = kEmpty64;
        }
    }
};

// the hardware's wrapping increment: returns the old value, stores
// old >= top ? 0 : old + 1
uint32_t atomic_inc_wrap(uint32_t* p, uint32_t top) {
    uint32_t old = peek(p);
    while (!__atomic_compare_exchange_n(p, &old, old >= top ? 0u : old + 1u, false, __ATOMIC_RELAXED,
                                        __ATOMIC_RELAXED)) {
    }
    return old;
}

bool bound_to(uint64_t* hdr_sig, uint64_t sig, uint64_t seen, bool designated, int mut) {
    if (mut == kNoSignature) return true;
    if (seen == sig) return true;
    if (seen == kEmpty64) {
        if (designated) publish(hdr_sig, sig);
        return true;
    }
    if (mut != kNoPoison) publish(hdr_sig, kSigPoisoned);
    return false;
}

// One call of the forward scan on workspace `ws` with layout signature
// `sig`.  Outputs h and idx are written by the tiles that run.
void diag_call(const DiagProblem& P, DiagWs& ws, uint64_t sig, Pool& pool, int mut, std::vector<float>& h,
               std::vector<int32_t>& idx) {
    const int64_t nt = ws.nt, nch = ws.nch, F = ws.F, L = ws.L, T = P.T, d = P.d, B = P.B, G = ws.groups;
    // grouped counters: the grid is padded to whole groups of G positions per
    // chain, and workgroup g = G i + x takes chain i mod nch, counter (chain, x)
    const int64_t grid = G > 1 ? (nt + G - 1) / G * G * nch : ws.ntiles;
    pool.launch(grid, [&](int64_t g, Rng& r) {
        const int64_t chain = G > 1 ? (g / G) % nch : (g % nch + g / nch) % nch;
        const int64_t grp = G > 1 ? g % G : 0;
        const uint64_t seen = peek(&ws.sig);
        const uint32_t per_call = (uint32_t)(G > 1 ? (nt + G - 1) / G : nt);
        const uint32_t top = mut == kWrapEveryCall ? per_call - 1u : 2u * per_call - 1u;
        const uint32_t old = atomic_inc_wrap(&ws.ctr[(size_t)(chain * G + grp)], top);
        const uint32_t t = old >= top ? 0u : old + 1u;
        const uint32_t n = t < per_call ? t : t - per_call;
        const uint32_t pos = (uint32_t)(n * G + grp);
        uint32_t bank = t < per_call ? 0u : 1u;
        if (mut == kOneBank) bank = 0;
        if (!bound_to(&ws.sig, sig, seen, chain == 0 && pos == 0, mut)) return;   // stand down
        if (pos >= (uint32_t)nt) return;   // grid padding (or a broken wrap; the result check catches it)
        jitter(r);
        const int64_t tile = pos, ticket = tile * nch + chain;
        const int64_t b = chain / ws.nfb, fb = chain % ws.nfb;
        const int64_t t0 = tile * L, t1 = std::min(T, t0 + L);
        auto begin_at = [&](int64_t t) { return t == 0 || P.start[(size_t)(b * T + t)] != 0; };
        std::vector<float> A((size_t)F, 1.0f), H((size_t)F, 0.0f);
        bool f = false;
        uint32_t c_tile = 0;
        for (int64_t t = t0; t < t1; ++t) {
            const bool bg = begin_at(t);
            f = f || bg;
            c_tile += bg ? 1u : 0u;
            for (int64_t v = 0; v < F; ++v) {
                const int64_t j = fb * F + v;
                if (j >= d) continue;
                const size_t o = (size_t)((b * T + t) * d + j);
                H[(size_t)v] = bg ? P.x[o] : std::fma(P.a[o], H[(size_t)v], P.x[o]);
                A[(size_t)v] = bg ? 1.0f : A[(size_t)v] * P.a[o];
            }
        }
        const uint32_t idle = bank ^ 1u;
        // publish the tile summary; clear this tile's words of the idle bank
        for (int64_t v = 0; v < F; ++v) {
            const size_t s = (size_t)(ticket * F + v);
            if (f) publish(&ws.incl[bank][s], fbits(canon(H[(size_t)v], mut)));
            else publish(&ws.agg[bank][s], pack2(A[(size_t)v], H[(size_t)v], mut));
            if (mut != kNoIdleClear && mut != kOneBank) {
                ws.agg[idle][s] = kEmpty64;
                ws.incl[idle][s] = kEmpty32;
            }
        }
        if (fb == 0) {
            if (mut != kNoIdleClear && mut != kOneBank) ws.cnt[idle][(size_t)(tile * B + b)] = kEmpty64;
            const bool incl_own = tile == 0 || mut == kCountOwnAsIncl;
            publish(&ws.cnt[bank][(size_t)(tile * B + b)], (incl_own ? kCountIncl : kCountOwn) | c_tile);
        }
        jitter(r);
        // look back for the carry of every feature
        std::vector<float> carry((size_t)F, 0.0f);
        if (!(t0 == 0 || P.start[(size_t)(b * T + t0)] != 0)) {
            for (int64_t v = 0; v < F; ++v) {
                float aA = 1.0f, aH = 0.0f;
                int64_t pred = ticket - nch;
                uint32_t polls = 0;
                while (true) {
                    const size_t s = (size_t)(pred * F + v);
                    const uint32_t wi = peek(&ws.incl[bank][s]);
                    if (wi != kEmpty32) {
                        carry[(size_t)v] = std::fma(aA, bitsf(wi), aH);
                        break;
                    }
                    const uint64_t wa = peek(&ws.agg[bank][s]);
                    if (wa != kEmpty64) {
                        aH = std::fma(aA, hi_of(wa), aH);
                        aA = aA * lo_of(wa);
                        pred -= nch;
                        polls = 0;
                        continue;
                    }
                    if (++polls > kMaxPolls) {
                        publish(&ws.timeout, 0u);
                        break;
                    }
                    if (polls % 64 == 0) std::this_thread::yield();
                }
            }
        }
        // begin count before the tile (episode index)
        uint32_t before = 0;
        if (fb == 0 && tile > 0) {
            int64_t k = tile - 1;
            uint32_t polls = 0;
            while (k >= 0) {
                const uint64_t w = peek(&ws.cnt[bank][(size_t)(k * B + b)]);
                if (w == kEmpty64) {
                    if (++polls > kMaxPolls) {
                        publish(&ws.timeout, 0u);
                        break;
                    }
                    if (polls % 64 == 0) std::this_thread::yield();
                    continue;
                }
                polls = 0;
                before += (uint32_t)(w & kCountValue);
                if (w & kCountIncl) break;
                --k;
            }
        }
        jitter(r);
        // the tile's inclusive prefix, then the outputs
        for (int64_t v = 0; v < F; ++v)
            if (!f) publish(&ws.incl[bank][(size_t)(ticket * F + v)],
                            fbits(canon(std::fma(A[(size_t)v], carry[(size_t)v], H[(size_t)v]), mut)));
        if (fb == 0 && tile > 0) publish(&ws.cnt[bank][(size_t)(tile * B + b)], kCountIncl | (before + c_tile));
        std::vector<float> hv = carry;
        uint32_t run = before;
        for (int64_t t = t0; t < t1; ++t) {
            const bool bg = begin_at(t);
            run += bg ? 1u : 0u;
            if (fb == 0) idx[(size_t)(b * T + t)] = (int32_t)run - 1;
            for (int64_t v = 0; v < F; ++v) {
                const int64_t j = fb * F + v;
                if (j >= d) continue;
                const size_t o = (size_t)((b * T + t) * d + j);
                hv[(size_t)v] = bg ? P.x[o] : std::fma(P.a[o], hv[(size_t)v], P.x[o]);
                h[o] = hv[(size_t)v];
            }
        }
    });
}

// largest conditioned error of h against the oracle, and whether the
// episode indices are exact (NaN-aware: NaN where the oracle has NaN)
bool diag_matches(const DiagProblem& P, const std::vector<float>& h, const std::vector<int32_t>& idx,
                  double* worst) {
    double w = 0.0;
    for (size_t i = 0; i < h.size(); ++i) {
        const double r = P.ref[i], y = h[i];
        if (r != r) {
            if (y == y) return false;
            continue;
        }
        if (y != y) return false;
        const double den = std::max(std::fabs(r), P.mag[i]);
        const double e = den > 0 ? std::fabs(y - r) / den : std::fabs(y - r);
        w = std::max(w, e);
    }
    *worst = w;
    for (size_t i = 0; i < idx.size(); ++i)
        if (idx[i] != P.idx[i]) return false;
    return w <= 1e-4;
}

bool load_diag(const std::string& dir, int k, DiagProblem& P) {
    FILE* f = std::fopen((dir + "/diag" + std::to_string(k) + ".shape").c_str(), "r");
    if (!f) return false;
    long long B, T, d;
    const int n = std::fscanf(f, "%lld %lld %lld", &B, &T, &d);
    std::fclose(f);
    if (n != 3) return false;
    P.B = B; P.T = T; P.d = d;
    const size_t N = (size_t)(B * T * d), BT = (size_t)(B * T);
    const std::string p = dir + "/diag" + std::to_string(k);
    return read_file(p + ".a", P.a, N) && read_file(p + ".x", P.x, N) && read_file(p + ".start", P.start, BT) &&
           read_file(p + ".ref", P.ref, N) && read_file(p + ".mag", P.mag, N) && read_file(p + ".idx", P.idx, BT);
}

// Calls on one prepared workspace: the three problems in turn, several
// rounds (each bank used repeatedly), every call checked against the oracle;
// then a call with another layout (another tile length) on the bound
// workspace, which must stand down and leave its outputs untouched, a call
// with the original layout that must stand down too (poisoned), and a new
// preparation after which the original layout computes again.
int run_diag(const std::string& dir, int schedules, int mut, bool grouped) {
    DiagProblem P[3];
    for (int k = 0; k < 3; ++k)
        if (!load_diag(dir, k, P[k])) {
            std::printf("cannot read problem %d\n", k);
            return 2;
        }
    int failures = 0;
    double worst = 0.0;
    for (int s = 0; s < schedules; ++s) {
        Rng r(0x5eed0000ull + (uint64_t)s);
        Pool pool(2 + (int)r.below(7), (uint64_t)s);
        const int64_t F = 1 + r.below(3), L = 4 + r.below(13);
        const DiagProblem& P0 = P[0];
        DiagWs ws;
        ws.groups = grouped ? 2 + (int64_t)r.below(7) : 1;
        ws.size_for(P0.B, P0.T, P0.d, F, L);
        ws.prepare();
        const uint64_t sig = 0x1234ull + (uint64_t)(F * 131 + L);
        bool ok = true;
        const int rounds = 2 + (int)r.below(2);
        for (int c = 0; c < 3 * rounds && ok; ++c) {
            const DiagProblem& Pk = P[c % 3];
            std::vector<float> h(Pk.ref.size(), std::nanf(""));
            std::vector<int32_t> idx(Pk.idx.size(), -99);
            diag_call(Pk, ws, sig, pool, mut, h, idx);
            double e = 0.0;
            if (ws.timeout != kEmpty32 || !diag_matches(Pk, h, idx, &e)) ok = false;
            worst = std::max(worst, e);
        }
        if (ok) {
            // another layout on the bound workspace: every tile stands down
            // (same memory, longer tiles: fewer tiles, so the arrays suffice)
            DiagWs other = ws;
            other.L = ws.L + 1;
            other.nt = (P0.T + other.L - 1) / other.L;
            other.ntiles = other.nt * other.nch;
            std::vector<float> h(P0.ref.size(), 7.0f);
            std::vector<int32_t> idx(P0.idx.size(), -7);
            diag_call(P0, other, sig + 1, pool, mut, h, idx);
            bool untouched = true;
            for (float v : h) untouched = untouched && v == 7.0f;
            if (!untouched || other.sig != kSigPoisoned) ok = false;
            // back to the first layout on the same (now poisoned) memory
            ws.sig = other.sig;
            ws.ctr = other.ctr;
            std::vector<float> h2(P0.ref.size(), 9.0f);
            diag_call(P0, ws, sig, pool, mut, h2, idx);
            bool untouched2 = true;
            for (float v : h2) untouched2 = untouched2 && v == 9.0f;
            if (!untouched2) ok = false;
            ws.prepare();
            std::vector<float> h3(P0.ref.size(), std::nanf(""));
            std::vector<int32_t> idx3(P0.idx.size(), -99);
            diag_call(P0, ws, sig, pool, mut, h3, idx3);
            double e = 0.0;
            if (ws.timeout != kEmpty32 || !diag_matches(P0, h3, idx3, &e)) ok = false;
        }
        if (!ok) {
            ++failures;
            if (mut != kNone) break;              // detected
        }
    }
    std::printf("diag%s mutation %d schedules %d failures %d worst_err %.3g\n", grouped ? " grouped" : "", mut,
                schedules, failures, worst);
    if (mut == kNone) return failures == 0 ? 0 : 1;
    return failures > 0 ? 0 : 1;
}

// ---------------------------------------------------------- discounted return
struct RetProblem {
    int64_t B = 0, T = 0;
    float gamma = 0.0f;
    std::vector<float> r;
    std::vector<uint8_t> start;
    std::vector<double> ref, mag;
};

struct RMap {
    float A, H;
    bool f;
};
RMap then(const RMap& left, const RMap& right) {   // left: earlier steps
    return RMap{left.A * right.A, left.f ? left.H : std::fma(left.A, right.H, left.H), left.f || right.f};
}
float apply(const RMap& m, float after) { return m.f ? m.H : std::fma(m.A, after, m.H); }

struct RetWs {
    int64_t nt = 0, L = 0, B = 0;
    uint64_t sig = kEmpty64;
    uint32_t timeout = kEmpty32;
    std::vector<uint32_t> epoch;          // [ticket]
    std::vector<uint64_t> agg[2], incl[2];
    void size_for(int64_t Bq, int64_t T, int64_t Lq) {
        B = Bq; L = Lq; nt = (T + L - 1) / L;
        epoch.assign((size_t)(B * nt), 0);
        for (int k = 0; k < 2; ++k) {
            agg[k].assign((size_t)(B * nt), 0);
            incl[k].assign((size_t)(B * nt), 0);
        }
    }
    void prepare() {
        sig = kEmpty64;
        timeout = kEmpty32;
        for (auto& e : epoch) e = kEmpty32;
        for (int k = 0; k < 2; ++k) {
            for (auto& w : agg[k]) w = kEmpty64;
            for (auto& w : incl[k]) w = kEmpty64;
        }
    }
};

// map of tile i (from the tape's start) of tape b, from its inputs
RMap tile_map(const RetProblem& P, int64_t b, int64_t i, int64_t L) {
    const int64_t t0 = i * L, t1 = std::min(P.T, t0 + L);
    RMap m{1.0f, 0.0f, false};
    for (int64_t t = t1 - 1; t >= t0; --t) {
        const bool end = t + 1 >= P.T || P.start[(size_t)(b * P.T + t + 1)] != 0;
        const RMap s{P.gamma, P.r[(size_t)(b * P.T + t)], end};
        m = then(s, m);
    }
    return m;
}

void ret_call(const RetProblem& P, RetWs& ws, uint64_t sig, Pool& pool, int mut, uint32_t fallback_polls,
              std::vector<float>& G) {
    const int64_t nt = ws.nt, B = P.B, L = ws.L;
    pool.launch(B * nt, [&](int64_t ticket, Rng& r) {
        const uint64_t seen = peek(&ws.sig);
        const int64_t j = ticket / B, b = ticket - j * B, i = nt - 1 - j;
        const uint32_t ep = ws.epoch[(size_t)ticket] + 1u;     // all ones reads as epoch 0
        uint32_t bank = ep & 1u;
        if (mut == kOneBank) bank = 0;
        if (!bound_to(&ws.sig, sig, seen, ticket == 0, mut)) return;
        const RMap TM = tile_map(P, b, i, L);
        const int64_t slot = b * nt + j;
        const uint32_t idle = bank ^ 1u;
        if (TM.f) publish(&ws.incl[bank][(size_t)slot], pack2(TM.H, 0.0f, mut));
        else publish(&ws.agg[bank][(size_t)slot], pack2(TM.H, TM.A, mut));
        if (mut != kNoIdleClear && mut != kOneBank) {
            ws.agg[idle][(size_t)slot] = kEmpty64;
            ws.incl[idle][(size_t)slot] = kEmpty64;
        }
        jitter(r);
        float carry = 0.0f;
        const int64_t t_next = (i + 1) * L;
        const bool need = j > 0 && P.start[(size_t)(b * P.T + t_next)] == 0;
        if (need) {
            RMap acc{1.0f, 0.0f, false};
            int64_t k = j - 1;
            uint32_t polls = 0, total = 0;
            while (true) {
                const uint64_t wi = peek(&ws.incl[bank][(size_t)(b * nt + k)]);
                if (wi != kEmpty64) {
                    carry = apply(acc, lo_of(wi));
                    break;
                }
                const uint64_t wa = peek(&ws.agg[bank][(size_t)(b * nt + k)]);
                if (wa != kEmpty64) {
                    acc = then(acc, RMap{hi_of(wa), lo_of(wa), false});
                    --k;
                    polls = 0;
                    continue;
                }
                if (++total > kMaxPolls) {
                    publish(&ws.timeout, 0u);
                    break;
                }
                if (++polls > fallback_polls) {
                    // the awaited tile has not published: its map from its inputs
                    const int64_t kk = mut == kFallbackWrongTile && k > 0 ? k - 1 : k;
                    const RMap M = tile_map(P, b, nt - 1 - kk, L);
                    acc = then(acc, M);
                    if (M.f) {
                        carry = acc.H;
                        break;
                    }
                    --k;
                    polls = 0;
                    continue;
                }
                if (polls % 16 == 0) std::this_thread::yield();
            }
        }
        if (!TM.f) publish(&ws.incl[bank][(size_t)slot], pack2(apply(TM, carry), 0.0f, mut));
        // outputs: walk the tile backwards from the carry
        float g = carry;
        const int64_t t0 = i * L, t1 = std::min(P.T, t0 + L);
        for (int64_t t = t1 - 1; t >= t0; --t) {
            const bool end = t + 1 >= P.T || P.start[(size_t)(b * P.T + t + 1)] != 0;
            g = end ? P.r[(size_t)(b * P.T + t)] : std::fma(P.gamma, g, P.r[(size_t)(b * P.T + t)]);
            G[(size_t)(b * P.T + t)] = g;
        }
        if (mut != kEpochNotStored) ws.epoch[(size_t)ticket] = ep;
    });
}

bool ret_matches(const RetProblem& P, const std::vector<float>& G, double* worst) {
    double w = 0.0;
    for (size_t i = 0; i < G.size(); ++i) {
        const double den = std::max(std::fabs(P.ref[i]), P.mag[i]);
        const double e = den > 0 ? std::fabs(G[i] - P.ref[i]) / den : std::fabs(G[i] - P.ref[i]);
        if (!(e <= 1e-4)) return false;
        w = std::max(w, e);
    }
    *worst = w;
    return true;
}

bool load_ret(const std::string& dir, int k, RetProblem& P) {
    FILE* f = std::fopen((dir + "/ret" + std::to_string(k) + ".shape").c_str(), "r");
    if (!f) return false;
    long long B, T;
    float gamma;
    const int n = std::fscanf(f, "%lld %lld %f", &B, &T, &gamma);
    std::fclose(f);
    if (n != 3) return false;
    P.B = B; P.T = T; P.gamma = gamma;
    const size_t N = (size_t)(B * T);
    const std::string p = dir + "/ret" + std::to_string(k);
    return read_file(p + ".r", P.r, N) && read_file(p + ".start", P.start, N) && read_file(p + ".ref", P.ref, N) &&
           read_file(p + ".mag", P.mag, N);
}

int run_return(const std::string& dir, int schedules, int mut) {
    RetProblem P[3];
    for (int k = 0; k < 3; ++k)
        if (!load_ret(dir, k, P[k])) {
            std::printf("cannot read return problem %d\n", k);
            return 2;
        }
    int failures = 0;
    double worst = 0.0;
    for (int s = 0; s < schedules; ++s) {
        Rng r(0xfeed0000ull + (uint64_t)s);
        Pool pool(2 + (int)r.below(7), (uint64_t)s);
        const int64_t L = 3 + r.below(14);
        // fallback after 0 .. 3 polls in a third of the schedules, else effectively never
        const uint32_t fb = r.below(3) == 0 ? r.below(4) : 1000000u;
        RetWs ws;
        ws.size_for(P[0].B, P[0].T, L);
        ws.prepare();
        const uint64_t sig = 0x777ull + (uint64_t)L;
        bool ok = true;
        const int rounds = 2 + (int)r.below(2);
        for (int c = 0; c < 3 * rounds && ok; ++c) {
            const RetProblem& Pk = P[c % 3];
            std::vector<float> G(Pk.ref.size(), std::nanf(""));
            ret_call(Pk, ws, sig, pool, mut, fb, G);
            double e = 0.0;
            if (ws.timeout != kEmpty32 || !ret_matches(Pk, G, &e)) ok = false;
            worst = std::max(worst, e);
        }
        if (!ok) {
            ++failures;
            if (mut != kNone) break;
        }
    }
    std::printf("return mutation %d schedules %d failures %d worst_err %.3g\n", mut, schedules, failures, worst);
    if (mut == kNone) return failures == 0 ? 0 : 1;
    return failures > 0 ? 0 : 1;
}

}  // namespace

int main(int argc, char** argv) {
    if (argc != 5) {
        std::printf("usage: %s <dir> diag|diag_grouped|return <schedules> <mutation>\n", argv[0]);
        return 2;
    }
    const std::string dir = argv[1], what = argv[2];
    const int schedules = std::atoi(argv[3]), mut = std::atoi(argv[4]);
    if (mut < 0 || mut >= kMutations) return 2;
    if (what == "diag") return run_diag(dir, schedules, mut, false);
    if (what == "diag_grouped") return run_diag(dir, schedules, mut, true);
    if (what == "return") return run_return(dir, schedules, mut);
    return 2;
}
