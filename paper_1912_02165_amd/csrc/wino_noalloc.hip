// wino_conv_run_noalloc (include/wino_conv.h): the fused convolution of
// wino_conv_run for callers that cannot allocate device memory (code under HIP
// graph capture, tight serving loops, harnesses that forbid hipMalloc).  It needs
// no plan: the scratch the fused path uses -- the transformed kernels, the split
// items' partial outputs and arrival counters, and a status word -- lives in a
// file-scope device array of fixed size, one copy per GPU, held until the process
// ends.  Every call on a GPU shares that GPU's copy, so calls that overlap on one
// GPU (on different streams, or from different threads) race.
#include "wino_conv.h"
#include "wino_internal.h"

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

namespace {

constexpr size_t kScratchBytes = WINO_NOALLOC_SCRATCH_BYTES;
constexpr size_t kAlign = 256;

// The scratch.  In host code its name is a host-side stand-in, not a device
// address: host code uses only the address hipGetSymbolAddress returns for the
// current device (g_dev below).
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
struct DeviceScratch {
    bool ready;
    unsigned char *ptr;  // the device address of `scratch` on this device
    int cus;             // compute units (persistent grid size)
};
std::mutex g_mu;
DeviceScratch g_dev[kMaxDevices];

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Once per device, with that device current: the scratch's device address.
int device_scratch(int dev, DeviceScratch *out) {
    if (dev < 0 || dev >= kMaxDevices) {
        wino::set_error("device %d: at most %d devices are supported", dev, kMaxDevices);
        return WINO_EUNSUPPORTED;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    DeviceScratch &d = g_dev[dev];
    if (!d.ready) {
        void *p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            wino::set_error("hipGetSymbolAddress of the scratch array: %s", hipGetErrorString(e));
            return WINO_EHIP;
        }
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) {
            (void)hipGetLastError();
            cus = 256;
        }
        d.ptr = static_cast<unsigned char *>(p);
        d.cus = cus;
        d.ready = true;
    }
    *out = d;
    return WINO_OK;
}

}  // namespace

extern "C" int wino_conv_run_noalloc(int N, int C, int K, int H, int W, int m, const float *x, const float *w,
                                     float *y, unsigned *status, void *stream) {
    wino::Geometry g;
    int rc = wino::make_geometry(N, C, K, H, W, m, WINO_ALGO_FUSED, &g);
    if (rc != WINO_OK) return rc;
    // transformed kernels, checked before any HIP call
    const size_t wt_bytes = (size_t)g.Kb_alloc * 16 * g.Cs * 4 * ((g.T2 + 3) / 4 * 4) * sizeof(float);
    if (align_up(wt_bytes) + kAlign > kScratchBytes) {
        wino::set_error("the transformed kernels take %zu bytes, the scratch of wino_conv_run_noalloc holds %zu "
                        "(C=%d K=%d m=%d); use a plan (wino_conv_plan) instead",
                        wt_bytes, kScratchBytes, C, K, m);
        return WINO_EUNSUPPORTED;
    }
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        wino::set_error("hipGetDevice: %s", hipGetErrorString(e));
        return WINO_EHIP;
    }
    DeviceScratch ds{};
    if ((rc = device_scratch(dev, &ds)) != WINO_OK) return rc;
    const wino::FusedCfg cfg = wino::fused_cfg_default(g, ds.cus);
    const wino::SplitInfo si = wino::fused_split_info(g, cfg);
    const size_t cnt_bytes = si.n_tail > 0 ? (size_t)si.n_tail * sizeof(unsigned) : 0;
    const size_t part_bytes = si.n_tail > 0 ? (size_t)si.n_tail * si.maxc * si.part_floats * sizeof(float) : 0;
    // layout: [status word | split counters | partial outputs | transformed kernels]
    const size_t off_cnt = kAlign, off_part = off_cnt + align_up(cnt_bytes);
    const size_t off_wt = off_part + align_up(part_bytes), total = off_wt + align_up(wt_bytes);
    if (total > kScratchBytes) {
        wino::set_error("this layer needs %zu bytes of scratch (transformed kernels %zu, partial outputs %zu), "
                        "wino_conv_run_noalloc holds %zu; use a plan (wino_conv_plan) instead",
                        total, wt_bytes, part_bytes, kScratchBytes);
        return WINO_EUNSUPPORTED;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t xb = (size_t)N * C * H * W * 4, yb = (size_t)N * K * H * W * 4, wb = (size_t)K * C * 9 * 4;
    if ((rc = wino::check_stream_device(s, dev)) != WINO_OK) return rc;
    if ((rc = wino::check_device_ptr(x, xb, dev, "x")) != WINO_OK) return rc;
    if ((rc = wino::check_device_ptr(w, wb, dev, "w")) != WINO_OK) return rc;
    if ((rc = wino::check_device_ptr(y, yb, dev, "y")) != WINO_OK) return rc;
    if (status && (rc = wino::check_device_ptr(status, sizeof(unsigned), dev, "status")) != WINO_OK) return rc;
    if (wino::overlap(x, xb, y, yb) || wino::overlap(w, wb, y, yb)) {
        wino::set_error("y overlaps x or w");
        return WINO_EINVAL;
    }
    unsigned char *base = ds.ptr;
    wino::SplitBuffers sb;
    sb.err = status ? status : reinterpret_cast<unsigned *>(base);
    sb.cnt = cnt_bytes ? reinterpret_cast<unsigned *>(base + off_cnt) : nullptr;
    sb.part = part_bytes ? reinterpret_cast<float *>(base + off_part) : nullptr;
    float *wt = reinterpret_cast<float *>(base + off_wt);
    // The kernel transform's first workgroup clears the scratch's status word and
    // the split counters (a kernel, not a memset, so a captured call replays it).
    e = wino::launch_weight_transform(g, w, wt, s, reinterpret_cast<unsigned *>(base),
                                      (int)((off_cnt + cnt_bytes) / sizeof(unsigned)));
    if (e != hipSuccess) {
        wino::set_error("kernel transform launch: %s", hipGetErrorString(e));
        return WINO_EHIP;
    }
    e = wino::launch_fused(g, cfg, x, wt, y, sb, s);
    if (e != hipSuccess) {
        wino::set_error("fused kernel launch: %s", hipGetErrorString(e));
        return WINO_EHIP;
    }
    return WINO_OK;
}
