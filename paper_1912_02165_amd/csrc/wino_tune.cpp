// Per-layer tuning of the tile size, the fused kernel's blocking (tiles and output
// channels per task) and optionally the algorithm, and the wisdom table that
// remembers the results (declared in include/wino_tune.h).
#include "wino_tune.h"
#include "wino_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

namespace {

using Key = std::tuple<std::string, int, int, int, int, int, int, unsigned>;  // arch, cus, N, C, K, H, W, mask
struct Choice {
    int m, algo;
    int R, kit;  // fused blocking (0 for the other algorithms)
    double us;
};

std::mutex g_mu;
std::map<Key, Choice> g_table;

// Tile sizes with fused blockings; F(7x7,3x3) runs three-stage only.
constexpr unsigned kFusedMBits = WINO_TUNE_M2 | WINO_TUNE_M4 | WINO_TUNE_M5 | WINO_TUNE_M6;
constexpr unsigned kMBits = kFusedMBits | WINO_TUNE_M7;
constexpr unsigned kAllBits = kMBits | WINO_TUNE_THREE_STAGE | WINO_TUNE_FFT;

// A mask is valid when it names at least one candidate: a fused tile size, the
// FFT-tile algorithm, or m = 7 together with the three-stage algorithm.
bool mask_ok(unsigned c) {
    if ((c & ~kAllBits) != 0) return false;
    return (c & (kFusedMBits | WINO_TUNE_FFT)) != 0 || ((c & WINO_TUNE_M7) && (c & WINO_TUNE_THREE_STAGE));
}

bool choice_ok(unsigned c, int m, int algo, int R, int kit) {
    if (algo == WINO_ALGO_FFT) return m == 14 && (c & WINO_TUNE_FFT) != 0 && R == 0 && kit == 0;
    if (m != 2 && m != 4 && m != 5 && m != 6 && m != 7) return false;
    if (!(c & (1u << m))) return false;
    if (algo == WINO_ALGO_THREE_STAGE) return (c & WINO_TUNE_THREE_STAGE) != 0 && R == 0 && kit == 0;
    return algo == WINO_ALGO_FUSED && wino::fused_blocking_built(m, R, kit);
}

// The plan of a choice: the fused blocking as an override.
wino_plan *plan_of(int N, int C, int K, int H, int W, const Choice &c) {
    wino_tuning t{};
    t.tiles_per_wg = c.R;
    t.k_per_wg = c.kit;
    return wino_conv_plan_ex(N, C, K, H, W, c.m, c.algo, c.algo == WINO_ALGO_FUSED ? &t : nullptr);
}

// Architecture name (up to the first ':' of gcnArchName) and compute units of the
// current device.
int device_key(std::string *arch, int *cus) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    hipDeviceProp_t prop;
    if (e == hipSuccess) e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        wino::set_error("hipGetDeviceProperties: %s", hipGetErrorString(e));
        return WINO_EHIP;
    }
    std::string a = prop.gcnArchName;
    *arch = a.substr(0, a.find(':'));
    *cus = prop.multiProcessorCount;
    return WINO_OK;
}

// Device buffers of one layer, filled with a constant, freed on destruction.
struct Buffers {
    float *x = nullptr, *w = nullptr, *y = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    ~Buffers() {
        if (x) (void)hipFree(x);
        if (w) (void)hipFree(w);
        if (y) (void)hipFree(y);
        if (e0) (void)hipEventDestroy(e0);
        if (e1) (void)hipEventDestroy(e1);
    }
    int alloc(size_t nx, size_t nw, size_t ny) {
        hipError_t e;
        if ((e = hipMalloc(&x, nx * 4)) != hipSuccess || (e = hipMalloc(&w, nw * 4)) != hipSuccess ||
            (e = hipMalloc(&y, ny * 4)) != hipSuccess) {
            (void)hipGetLastError();
            wino::set_error("tuning buffers: device allocation failed (%s)", hipGetErrorString(e));
            return WINO_ENOMEM;
        }
        const unsigned v = 0x3c23d70au;  // 0.01f
        if ((e = hipMemsetD32(reinterpret_cast<hipDeviceptr_t>(x), (int)v, nx)) != hipSuccess ||
            (e = hipMemsetD32(reinterpret_cast<hipDeviceptr_t>(w), (int)v, nw)) != hipSuccess ||
            (e = hipEventCreate(&e0)) != hipSuccess || (e = hipEventCreate(&e1)) != hipSuccess) {
            (void)hipGetLastError();
            wino::set_error("tuning buffers: %s", hipGetErrorString(e));
            return WINO_EHIP;
        }
        return WINO_OK;
    }
};

// GPU time (microseconds) per call of n back-to-back calls of the pretransformed
// path, between two events on the default stream.
int time_batch(wino_plan *p, const Buffers &b, int n, double *us) {
    hipError_t e = hipEventRecord(b.e0, nullptr);
    int st = WINO_OK;
    for (int i = 0; e == hipSuccess && st == WINO_OK && i < n; ++i) st = wino_conv_run_pretransformed(p, b.x, b.y, nullptr);
    if (st != WINO_OK) return st;
    if (e == hipSuccess) e = hipEventRecord(b.e1, nullptr);
    if (e == hipSuccess) e = hipEventSynchronize(b.e1);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, b.e0, b.e1);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        wino::set_error("tuning: timing failed (%s)", hipGetErrorString(e));
        return WINO_EHIP;
    }
    *us = ms * 1e3 / n;
    return WINO_OK;
}

// Time per call (microseconds) of the plan: its kernels transformed, then at
// least kWarmUs of back-to-back calls (the shader clock needs tens of
// milliseconds of work to reach its working frequency, so without this the first
// candidates would be timed at a lower clock than the later ones), then the
// median of 5 batches of back-to-back calls of at least kBatchUs each.
constexpr double kWarmUs = 20000.0, kBatchUs = 1000.0;
int time_plan(wino_plan *p, const Buffers &b, double *us) {
    int st = wino_conv_set_weights(p, b.w, nullptr);
    if (st != WINO_OK) return st;
    double per = 0.0, warm = 0.0;
    int n = 4;
    for (int it = 0; warm < kWarmUs && it < 1000; ++it) {  // bounded even if a batch times as 0
        if ((st = time_batch(p, b, n, &per)) != WINO_OK) return st;
        warm += per * n;
        if (n < 256 && per * n < kBatchUs) n *= 2;
    }
    n = per > 0.0 ? (int)(kBatchUs / per) + 1 : 1;
    std::vector<double> t(5);
    for (double &v : t)
        if ((st = time_batch(p, b, n, &v)) != WINO_OK) return st;
    std::sort(t.begin(), t.end());
    *us = t[t.size() / 2];
    return WINO_OK;
}

}  // namespace

wino_plan *wino_conv_plan_tuned(int N, int C, int K, int H, int W, unsigned candidates, int *chosen_m,
                                int *chosen_algo, double *call_us) {
    if (N < 1 || C < 1 || K < 1 || H < 1 || W < 1) {
        wino::set_error("sizes must be >= 1 (N=%d C=%d K=%d H=%d W=%d)", N, C, K, H, W);
        return nullptr;
    }
    if (!mask_ok(candidates)) {
        wino::set_error("candidate mask 0x%x: needs a WINO_TUNE_M2/4/5/6 or WINO_TUNE_FFT bit, or WINO_TUNE_M7 "
                        "with WINO_TUNE_THREE_STAGE, and no other bits",
                        candidates);
        return nullptr;
    }
    std::string arch;
    int cus = 0;
    if (device_key(&arch, &cus) != WINO_OK) return nullptr;
    const Key key{arch, cus, N, C, K, H, W, candidates};
    Choice best{0, 0, 0, 0, 0.0};
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_table.find(key);
        if (it != g_table.end()) best = it->second;
    }
    if (best.m == 0) {
        // candidates: per tile size every built fused blocking, the three-stage
        // algorithm if asked for, and the FFT-tile algorithm if asked for
        std::vector<Choice> cands;
        for (int m : {2, 4, 5, 6, 7}) {
            if (!(candidates & (1u << m))) continue;
            for (const wino::FusedBlocking &b : wino::kFusedBlockings)
                if (b.m == m) cands.push_back(Choice{m, WINO_ALGO_FUSED, b.R, b.kit, 0.0});
            if (candidates & WINO_TUNE_THREE_STAGE) cands.push_back(Choice{m, WINO_ALGO_THREE_STAGE, 0, 0, 0.0});
        }
        if (candidates & WINO_TUNE_FFT) cands.push_back(Choice{14, WINO_ALGO_FFT, 0, 0, 0.0});
        Buffers b;
        bool have_buffers = false;
        for (Choice c : cands) {
            wino_plan *p = plan_of(N, C, K, H, W, c);
            if (!p) return nullptr;  // message set by the constructor
            if (!have_buffers) {
                if (b.alloc((size_t)N * C * H * W, (size_t)K * C * 9, (size_t)N * K * H * W) != WINO_OK) {
                    wino_conv_destroy(p);
                    return nullptr;
                }
                have_buffers = true;
            }
            const int st = time_plan(p, b, &c.us);
            wino_conv_destroy(p);
            if (st != WINO_OK) return nullptr;
            if (best.m == 0 || c.us < best.us) best = c;
        }
        std::lock_guard<std::mutex> lk(g_mu);
        g_table[key] = best;
    }
    wino_plan *p = plan_of(N, C, K, H, W, best);
    if (!p) return nullptr;
    if (chosen_m) *chosen_m = best.m;
    if (chosen_algo) *chosen_algo = best.algo;
    if (call_us) *call_us = best.us;
    return p;
}

int wino_wisdom_lookup(const char *arch, int cus, int N, int C, int K, int H, int W, unsigned candidates,
                       int *found, int *m, int *algo, int *tiles_per_wg, int *k_per_wg) {
    if (!arch || !found || !m || !algo || !tiles_per_wg || !k_per_wg) {
        wino::set_error("wino_wisdom_lookup: NULL argument");
        return WINO_EINVAL;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_table.find(Key{arch, cus, N, C, K, H, W, candidates});
    *found = it != g_table.end() ? 1 : 0;
    if (*found) {
        *m = it->second.m;
        *algo = it->second.algo;
        *tiles_per_wg = it->second.R;
        *k_per_wg = it->second.kit;
    }
    return WINO_OK;
}

int wino_wisdom_save(const char *path) {
    if (!path) {
        wino::set_error("wino_wisdom_save: NULL path");
        return WINO_EINVAL;
    }
    FILE *f = fopen(path, "w");
    if (!f) {
        wino::set_error("wino_wisdom_save: cannot write %s", path);
        return WINO_EINVAL;
    }
    fprintf(f, "# winograd wisdom: arch cus N C K H W candidates m algo tiles_per_wg k_per_wg microseconds\n");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        for (const auto &kv : g_table) {
            const Key &k = kv.first;
            fprintf(f, "%s %d %d %d %d %d %d 0x%x %d %d %d %d %.3f\n", std::get<0>(k).c_str(), std::get<1>(k),
                    std::get<2>(k), std::get<3>(k), std::get<4>(k), std::get<5>(k), std::get<6>(k),
                    std::get<7>(k), kv.second.m, kv.second.algo, kv.second.R, kv.second.kit, kv.second.us);
        }
    }
    if (fclose(f) != 0) {
        wino::set_error("wino_wisdom_save: error writing %s", path);
        return WINO_EINVAL;
    }
    return WINO_OK;
}

int wino_wisdom_load(const char *path) {
    if (!path) {
        wino::set_error("wino_wisdom_load: NULL path");
        return WINO_EINVAL;
    }
    FILE *f = fopen(path, "r");
    if (!f) {
        wino::set_error("wino_wisdom_load: cannot read %s", path);
        return WINO_EINVAL;
    }
    std::vector<std::pair<Key, Choice>> entries;
    char line[512];
    int lineno = 0;
    int st = WINO_OK;
    while (fgets(line, sizeof line, f)) {
        ++lineno;
        const size_t len = strlen(line);
        if (len == sizeof line - 1 && line[len - 1] != '\n') {
            wino::set_error("wino_wisdom_load: %s:%d: line too long", path, lineno);
            st = WINO_EINVAL;
            break;
        }
        const char *s = line;
        while (*s == ' ' || *s == '\t') ++s;
        if (*s == '#' || *s == '\n' || *s == '\r' || *s == '\0') continue;
        char arch[64];
        int cus, N, C, K, H, W, m, algo, R, kit, used = 0;
        unsigned cand;
        double us;
        const int n = sscanf(s, "%63s %d %d %d %d %d %d %x %d %d %d %d %lf %n", arch, &cus, &N, &C, &K, &H, &W,
                             &cand, &m, &algo, &R, &kit, &us, &used);
        if (n != 13 || s[used] != '\0' || cus < 1 || N < 1 || C < 1 || K < 1 || H < 1 || W < 1 ||
            !mask_ok(cand) || !choice_ok(cand, m, algo, R, kit) || !(us >= 0.0)) {
            wino::set_error("wino_wisdom_load: %s:%d: malformed entry", path, lineno);
            st = WINO_EINVAL;
            break;
        }
        entries.push_back({Key{arch, cus, N, C, K, H, W, cand}, Choice{m, algo, R, kit, us}});
    }
    fclose(f);
    if (st != WINO_OK) return st;
    std::lock_guard<std::mutex> lk(g_mu);
    for (const auto &e : entries) g_table[e.first] = e.second;
    return WINO_OK;
}

void wino_wisdom_clear(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_table.clear();
}

int wino_wisdom_size(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    return (int)g_table.size();
}
