/*
 * wsr_api.cpp - the C ABI of libwsr (declared in include/wsr.h): argument checks, error reporting,
 * the host-range registry and launch orchestration.  Every check runs before anything is enqueued,
 * so a rejected call leaves the stream untouched.  Argument checks make no HIP call.
 */
#include <hip/hip_runtime_api.h>
#include <sys/mman.h>
#include <unistd.h>

#include <algorithm>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <thread>
#include <vector>

#include "wsr.h"
#include "wsr_copy.h"
#include "wsr_internal.h"
#include "wsr_mma_launch.h"

using wsr::DevMat;

namespace {

thread_local char g_err[512] = "";

wsr_status fail(wsr_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

wsr_status ok() {
    g_err[0] = '\0';
    return WSR_OK;
}

wsr_status hip_fail(hipError_t e, const char* what) {
    return fail(WSR_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

/* a * b * c without overflow of int64 (all arguments >= 0). */
bool mul_fits(int64_t a, int64_t b, int64_t c = 1) {
    const __int128 r = (__int128)a * b * c;
    return r <= INT64_MAX;
}

struct Reg {
    size_t bytes;
    void* dev;
    bool pinned_here;
};
std::mutex g_mu;
std::map<uintptr_t, Reg> g_reg;

/* Shared validation of one matrix (standalone GEMV or sweep entry). */
wsr_status check_matrix(int fmt, int64_t M, int64_t K, const void* w, const void* scales,
                        const void* x, const float* y, const char* who) {
    if (fmt != WSR_F16 && fmt != WSR_BF16 && fmt != WSR_Q4 && fmt != WSR_I8)
        return fail(WSR_E_ARG, "%s: unknown format %d", who, fmt);
    if (M < 0 || K < 0) return fail(WSR_E_ARG, "%s: negative size M=%lld K=%lld", who, (long long)M, (long long)K);
    if (!mul_fits(M, K, 2)) return fail(WSR_E_SIZE, "%s: M*K overflows", who);
    const int kq = fmt == WSR_Q4 ? 32 : fmt == WSR_I8 ? 16 : 8;
    if (K % kq != 0) return fail(WSR_E_ALIGN, "%s: K=%lld must be a multiple of %d", who, (long long)K, kq);
    if (M == 0) return WSR_OK;
    if (!w || !x || !y) return fail(WSR_E_ARG, "%s: null weight, activation or output pointer", who);
    if ((fmt == WSR_Q4 || fmt == WSR_I8) && !scales) return fail(WSR_E_ARG, "%s: q4 and int8 need scales", who);
    if (!aligned(w, 16) || !aligned(x, 16))
        return fail(WSR_E_ALIGN, "%s: weights and activations must be 16-byte aligned", who);
    if (!aligned(y, 4)) return fail(WSR_E_ALIGN, "%s: output must be 4-byte aligned", who);
    if ((fmt == WSR_Q4 || fmt == WSR_I8) && !aligned(scales, 2))
        return fail(WSR_E_ALIGN, "%s: scales must be 2-byte aligned", who);
    return WSR_OK;
}

DevMat make_devmat(int fmt, int64_t M, int64_t K, const void* w, const void* scales, const void* x,
                   float* y) {
    DevMat d{};
    d.w = w;
    d.s = (fmt == WSR_Q4 || fmt == WSR_I8) ? scales : nullptr;
    d.x = x;
    d.y = y;
    d.M = M;
    d.fmt = fmt;
    if (fmt == WSR_Q4) {
        d.nc = K / 32;
        d.row_bytes = K / 2 + (K / 32) * 2;
    } else if (fmt == WSR_I8) {
        d.nc = K / 16;
        d.row_bytes = K + 2;                         /* codes plus the row's scale */
    } else {
        d.nc = K / 8;
        d.row_bytes = K * 2;
    }
    if (d.row_bytes == 0) d.row_bytes = 1;   /* K = 0: rows still need an owner to write y = 0 */
    return d;
}

/* [p, p + bytes) lies inside [start, start + size). */
bool inside(const void* p, size_t bytes, const void* start, size_t size) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(p), s0 = reinterpret_cast<uintptr_t>(start);
    return a >= s0 && a - s0 <= size && bytes <= size - (a - s0);
}

/* Whether the pinned allocation that holds `host` (device view `dev`) covers [host, host + bytes):
 * 1 yes, 0 the range runs past its end, -1 the runtime reports no extent.  The runtime is asked for
 * the allocation's range through the host address and, if that gives no answer, through the device
 * address.  *start and *size receive the extent found (for messages). */
int pinned_extent_covers(const void* host, const void* dev, size_t bytes, const void** start_out, size_t* size_out) {
    void* start = nullptr;
    size_t size = 0;
    hipDeviceptr_t hp = const_cast<void*>(host);
    if (hipPointerGetAttribute(&start, HIP_POINTER_ATTRIBUTE_RANGE_START_ADDR, hp) == hipSuccess &&
        hipPointerGetAttribute(&size, HIP_POINTER_ATTRIBUTE_RANGE_SIZE, hp) == hipSuccess && size > 0 &&
        inside(host, 1, start, size)) {
        *start_out = start;
        *size_out = size;
        return inside(host, bytes, start, size) ? 1 : 0;
    }
    (void)hipGetLastError();
    hipDeviceptr_t base = nullptr;
    size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void*>(dev)) == hipSuccess && size > 0 &&
        inside(dev, 1, base, size)) {
        *start_out = base;
        *size_out = size;
        return inside(dev, bytes, base, size) ? 1 : 0;
    }
    (void)hipGetLastError();
    return -1;
}

/* The extent of the pinned allocation that holds `host` must cover the whole requested range; a
 * range the runtime cannot bound is refused. */
wsr_status check_pinned_extent(const void* host, const void* dev, size_t bytes) {
    const void* start = nullptr;
    size_t size = 0;
    const int c = pinned_extent_covers(host, dev, bytes, &start, &size);
    if (c == 1) return WSR_OK;
    if (c == 0)
        return fail(WSR_E_SIZE, "register_host: %p + %zu runs past the end of its pinned allocation "
                    "(%p + %zu)", host, bytes, start, size);
    return fail(WSR_E_UNSUPPORTED, "register_host: the runtime does not report the extent of the pinned "
                "allocation holding %p, so the range cannot be checked", host);
}

}  // namespace

extern "C" {

const char* wsr_last_error(void) { return g_err; }

int wsr_abi_version(void) { return WSR_ABI_VERSION; }

/* ---------------------------------- host ranges -------------------------------------------- */

wsr_status wsr_register_host(const void* host, size_t bytes, unsigned flags, const void** dev_out,
                             unsigned* granted_out) {
    if (!host || !dev_out) return fail(WSR_E_ARG, "register_host: null pointer");
    if (bytes == 0) return fail(WSR_E_ARG, "register_host: empty range");
    if (flags & ~(WSR_REG_READONLY | WSR_REG_PIN)) return fail(WSR_E_ARG, "register_host: unknown flags %#x", flags);
    const long page = sysconf(_SC_PAGESIZE);
    if (!aligned(host, (uintptr_t)page) || bytes % (size_t)page != 0)
        return fail(WSR_E_ALIGN, "register_host: base %p and length %zu must be multiples of the page size %ld",
                    host, bytes, page);
    std::lock_guard<std::mutex> lk(g_mu);
    const uintptr_t key = reinterpret_cast<uintptr_t>(host);
    if (g_reg.count(key)) return fail(WSR_E_STATE, "register_host: %p is already registered", host);

    unsigned granted = 0;
    void* dev = nullptr;
    bool pinned_here = false;
    hipPointerAttribute_t attr{};
    const hipError_t qa = hipPointerGetAttributes(&attr, host);
    if (qa == hipSuccess && attr.type == hipMemoryTypeHost && attr.devicePointer != nullptr) {
        /* Already pinned and mapped: adopt in place, but only if the whole range lies inside that
         * one pinned allocation; pages past its end are not device-visible. */
        const wsr_status st = check_pinned_extent(host, attr.devicePointer, bytes);
        if (st != WSR_OK) return st;
        dev = attr.devicePointer;
        granted |= WSR_REG_PREPINNED;
    } else {
        (void)hipGetLastError();                /* an unknown pointer is not an error here */
        if (!(flags & WSR_REG_PIN))
            return fail(WSR_E_UNSUPPORTED,
                        "register_host: %p is not device-visible host memory (pass WSR_REG_PIN to pin it)", host);
        void* h = const_cast<void*>(host);
        hipError_t e = hipErrorNotSupported;
        if (flags & WSR_REG_READONLY) {
            e = hipHostRegister(h, bytes, hipHostRegisterMapped | hipHostRegisterReadOnly);
            if (e == hipSuccess) granted |= WSR_REG_READONLY;
            else (void)hipGetLastError();
        }
        if (e != hipSuccess) e = hipHostRegister(h, bytes, hipHostRegisterMapped);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(WSR_E_UNSUPPORTED, "register_host: the runtime refused to pin %p (+%zu): %s", host,
                        bytes, hipGetErrorString(e));
        }
        pinned_here = true;
        e = hipHostGetDevicePointer(&dev, h, 0);
        if (e != hipSuccess) {
            (void)hipHostUnregister(h);
            return hip_fail(e, "register_host: hipHostGetDevicePointer");
        }
    }
    g_reg[key] = Reg{bytes, dev, pinned_here};
    *dev_out = dev;
    if (granted_out) *granted_out = granted;
    return ok();
}

wsr_status wsr_unregister_host(const void* host) {
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_reg.find(reinterpret_cast<uintptr_t>(host));
    if (it == g_reg.end()) return fail(WSR_E_STATE, "unregister_host: %p is not registered", host);
    if (it->second.pinned_here) {
        const hipError_t e = hipHostUnregister(const_cast<void*>(host));
        if (e != hipSuccess) return hip_fail(e, "unregister_host: hipHostUnregister");
    }
    g_reg.erase(it);
    return ok();
}

/* ---------------------------------- probe --------------------------------------------------- */

size_t wsr_probe_workspace_bytes(size_t n) {
    return 8 * (size_t)wsr::probe_grid((int64_t)n);
}

wsr_status wsr_probe_read(const float* buf, size_t n, double* sum_dev, void* ws, size_t ws_bytes,
                          void* stream) {
    if (n > (size_t)INT64_MAX / 4) return fail(WSR_E_SIZE, "probe_read: n too large");
    if ((n && !buf) || !sum_dev || !ws) return fail(WSR_E_ARG, "probe_read: null pointer");
    if (!aligned(buf, 16) || !aligned(ws, 16) || !aligned(sum_dev, 8))
        return fail(WSR_E_ALIGN, "probe_read: buf and ws must be 16-byte and sum_dev 8-byte aligned");
    const size_t need = wsr_probe_workspace_bytes(n);
    if (ws_bytes < need) return fail(WSR_E_SIZE, "probe_read: workspace %zu < %zu bytes", ws_bytes, need);
    const hipError_t e = wsr::launch_probe(buf, (int64_t)n, sum_dev, ws, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "probe_read: launch");
    return ok();
}

/* ---------------------------------- GEMVs --------------------------------------------------- */

wsr_status wsr_gemv_f16(const void* W, const void* x, float* y, int64_t M, int64_t K, int fmt,
                        void* stream) {
    if (fmt != WSR_F16 && fmt != WSR_BF16) return fail(WSR_E_ARG, "gemv_f16: format must be WSR_F16 or WSR_BF16");
    wsr_status st = check_matrix(fmt, M, K, W, nullptr, x, y, "gemv_f16");
    if (st != WSR_OK) return st;
    if (M == 0) return ok();
    const hipError_t e = wsr::launch_gemv(make_devmat(fmt, M, K, W, nullptr, x, y), static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gemv_f16: launch");
    return ok();
}

wsr_status wsr_gemv_f16_cols(const void* W, const void* x, int64_t x_col_stride, float* y,
                             int64_t y_col_stride, int64_t M, int64_t K, int32_t T, int fmt, void* stream) {
    if (fmt != WSR_F16 && fmt != WSR_BF16)
        return fail(WSR_E_ARG, "gemv_f16_cols: format must be WSR_F16 or WSR_BF16");
    if (T != 1 && T != 2 && T != 4 && T != 8 && T != 16)
        return fail(WSR_E_ARG, "gemv_f16_cols: T=%d must be 1, 2, 4, 8 or 16", T);
    wsr_status st = check_matrix(fmt, M, K, W, nullptr, x, y, "gemv_f16_cols");
    if (st != WSR_OK) return st;
    if (x_col_stride < 0 || x_col_stride % 16 || y_col_stride < 0 || y_col_stride % 4)
        return fail(WSR_E_ALIGN, "gemv_f16_cols: column strides must be >= 0 and multiples of 16 (x) and 4 (y)");
    if (T > 1 && y_col_stride < M * 4)
        return fail(WSR_E_ARG, "gemv_f16_cols: output columns overlap (y_col_stride %lld < 4 M)",
                    (long long)y_col_stride);
    if (!mul_fits(x_col_stride, T) || !mul_fits(y_col_stride, T))
        return fail(WSR_E_SIZE, "gemv_f16_cols: column strides overflow");
    if (M == 0) return ok();
    DevMat d = make_devmat(fmt, M, K, W, nullptr, x, y);
    d.x_stride = x_col_stride;
    d.y_stride = y_col_stride;
    const hipError_t e = wsr::launch_gemv_cols(d, T, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gemv_f16_cols: launch");
    return ok();
}

wsr_status wsr_gemv_q4_cols(const uint8_t* Wq, const uint16_t* scales, const uint16_t* x,
                            int64_t x_col_stride, float* y, int64_t y_col_stride, int64_t M, int64_t K,
                            int32_t T, void* stream) {
    if (T != 1 && T != 2 && T != 4 && T != 8)
        return fail(WSR_E_ARG, "gemv_q4_cols: T=%d must be 1, 2, 4 or 8", T);
    wsr_status st = check_matrix(WSR_Q4, M, K, Wq, scales, x, y, "gemv_q4_cols");
    if (st != WSR_OK) return st;
    if (x_col_stride < 0 || x_col_stride % 16 || y_col_stride < 0 || y_col_stride % 4)
        return fail(WSR_E_ALIGN, "gemv_q4_cols: column strides must be >= 0 and multiples of 16 (x) and 4 (y)");
    if (T > 1 && y_col_stride < M * 4)
        return fail(WSR_E_ARG, "gemv_q4_cols: output columns overlap (y_col_stride %lld < 4 M)",
                    (long long)y_col_stride);
    if (!mul_fits(x_col_stride, T) || !mul_fits(y_col_stride, T))
        return fail(WSR_E_SIZE, "gemv_q4_cols: column strides overflow");
    if (M == 0) return ok();
    DevMat d = make_devmat(WSR_Q4, M, K, Wq, scales, x, y);
    d.x_stride = x_col_stride;
    d.y_stride = y_col_stride;
    const hipError_t e = wsr::launch_gemv_cols(d, T, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gemv_q4_cols: launch");
    return ok();
}

wsr_status wsr_gemv_i8(const int8_t* Wq, const uint16_t* scales, const uint16_t* x, float* y,
                       int64_t M, int64_t K, void* stream) {
    wsr_status st = check_matrix(WSR_I8, M, K, Wq, scales, x, y, "gemv_i8");
    if (st != WSR_OK) return st;
    if (M == 0) return ok();
    const hipError_t e = wsr::launch_gemv(make_devmat(WSR_I8, M, K, Wq, scales, x, y), static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gemv_i8: launch");
    return ok();
}

wsr_status wsr_gemv_i8_cols(const int8_t* Wq, const uint16_t* scales, const uint16_t* x,
                            int64_t x_col_stride, float* y, int64_t y_col_stride, int64_t M, int64_t K,
                            int32_t T, void* stream) {
    if (T != 1 && T != 2 && T != 4 && T != 8)
        return fail(WSR_E_ARG, "gemv_i8_cols: T=%d must be 1, 2, 4 or 8", T);
    wsr_status st = check_matrix(WSR_I8, M, K, Wq, scales, x, y, "gemv_i8_cols");
    if (st != WSR_OK) return st;
    if (x_col_stride < 0 || x_col_stride % 16 || y_col_stride < 0 || y_col_stride % 4)
        return fail(WSR_E_ALIGN, "gemv_i8_cols: column strides must be >= 0 and multiples of 16 (x) and 4 (y)");
    if (T > 1 && y_col_stride < M * 4)
        return fail(WSR_E_ARG, "gemv_i8_cols: output columns overlap (y_col_stride %lld < 4 M)",
                    (long long)y_col_stride);
    if (!mul_fits(x_col_stride, T) || !mul_fits(y_col_stride, T))
        return fail(WSR_E_SIZE, "gemv_i8_cols: column strides overflow");
    if (M == 0) return ok();
    DevMat d = make_devmat(WSR_I8, M, K, Wq, scales, x, y);
    d.x_stride = x_col_stride;
    d.y_stride = y_col_stride;
    const hipError_t e = wsr::launch_gemv_cols(d, T, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gemv_i8_cols: launch");
    return ok();
}

wsr_status wsr_gemv_q4(const uint8_t* Wq, const uint16_t* scales, const uint16_t* x, float* y,
                       int64_t M, int64_t K, void* stream) {
    wsr_status st = check_matrix(WSR_Q4, M, K, Wq, scales, x, y, "gemv_q4");
    if (st != WSR_OK) return st;
    if (M == 0) return ok();
    const hipError_t e = wsr::launch_gemv(make_devmat(WSR_Q4, M, K, Wq, scales, x, y), static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gemv_q4: launch");
    return ok();
}

/* ---------------------------------- decode sweep -------------------------------------------- */

size_t wsr_sweep_workspace_bytes(const wsr_mat* mats, int32_t n) {
    (void)mats;
    if (n <= 0) return 0;
    return wsr::SWEEP_CTR_BYTES + ((size_t)n * sizeof(DevMat) + 255) / 256 * 256 +
           ((size_t)n * sizeof(int64_t) + 255) / 256 * 256;
}

}  // extern "C"

namespace {

struct Seg {
    int first, count, fmt;
    int64_t total;
};

/* A checked sweep: the device table and the launch groups (segments between
   WSR_MAT_AFTER_PREVIOUS flags). */
struct SweepPlan {
    std::vector<DevMat> tab;
    std::vector<Seg> segs;
    int32_t batch = 1;
};

wsr_status plan_table(const wsr_mat* mats, int32_t n, int32_t batch, int32_t n_tokens, SweepPlan& p);

/* Every check of a sweep with a caller's workspace; enqueues nothing. */
wsr_status plan_sweep(const wsr_mat* mats, int32_t n, int32_t n_tokens, int32_t batch, void* ws,
                      size_t ws_bytes, SweepPlan& p) {
    if (n < 0 || n_tokens < 1) return fail(WSR_E_ARG, "decode_sweep: n=%d n_tokens=%d", n, n_tokens);
    if (batch != 1 && batch != 2 && batch != 4 && batch != 8 && batch != 16)
        return fail(WSR_E_ARG, "decode_sweep: batch=%d must be 1, 2, 4, 8 or 16", batch);
    if (n == 0) return ok();
    if (!mats || !ws) return fail(WSR_E_ARG, "decode_sweep: null pointer");
    if (!aligned(ws, 256)) return fail(WSR_E_ALIGN, "decode_sweep: workspace must be 256-byte aligned");
    const size_t need = wsr_sweep_workspace_bytes(mats, n);
    if (ws_bytes < need) return fail(WSR_E_SIZE, "decode_sweep: workspace %zu < %zu bytes", ws_bytes, need);
    return plan_table(mats, n, batch, n_tokens, p);
}

/* The per-matrix checks and the device table of a sweep (n > 0, mats not null). */
wsr_status plan_table(const wsr_mat* mats, int32_t n, int32_t batch, int32_t n_tokens, SweepPlan& p) {
    p.tab.assign((size_t)n, DevMat{});
    p.segs.clear();
    char who[64];
    for (int32_t i = 0; i < n; ++i) {
        const wsr_mat& m = mats[i];
        std::snprintf(who, sizeof who, "decode_sweep: matrix %d", i);
        wsr_status st = check_matrix(m.fmt, m.M, m.K, m.w, m.scales, m.x, m.y, who);
        if (st != WSR_OK) return st;
        if (m.flags & ~WSR_MAT_AFTER_PREVIOUS) return fail(WSR_E_ARG, "%s: unknown flags %#x", who, m.flags);
        if (m.x_tok_stride < 0 || m.y_tok_stride < 0 || m.x_tok_stride % 16 || m.y_tok_stride % 4)
            return fail(WSR_E_ALIGN, "%s: token strides must be >= 0 and multiples of 16 (x) and 4 (y)", who);
        if (!mul_fits(m.x_tok_stride, n_tokens) || !mul_fits(m.y_tok_stride, n_tokens))
            return fail(WSR_E_SIZE, "%s: token strides overflow", who);
        if (batch > 1 && m.M > 0 && m.y_tok_stride < m.M * 4)
            return fail(WSR_E_ARG, "%s: tokens of one pass would share outputs (y_tok_stride < 4 M)", who);
        if (p.segs.empty() || (m.flags & WSR_MAT_AFTER_PREVIOUS)) p.segs.push_back(Seg{i, 0, m.fmt, 0});
        Seg& g = p.segs.back();
        DevMat d = make_devmat(m.fmt, m.M, m.K, m.w, m.scales, m.x, m.y);
        d.x_stride = m.x_tok_stride;
        d.y_stride = m.y_tok_stride;
        d.cost0 = g.total;
        if (!mul_fits(d.M, d.row_bytes) || g.total > INT64_MAX / 4 - d.M * d.row_bytes)
            return fail(WSR_E_SIZE, "%s: weight stream too large", who);
        g.total += d.M * d.row_bytes;
        if (g.fmt != m.fmt) g.fmt = 0;
        g.count += 1;
        p.tab[(size_t)i] = d;
    }
    /* Passes of `batch` tokens, at most 8 when the table holds q4 or int8 matrices. */
    for (int32_t i = 0; i < n && batch > 8; ++i)
        if (mats[i].fmt == WSR_Q4 || mats[i].fmt == WSR_I8) batch = 8;
    p.batch = batch;
    return ok();
}

/* Enqueue a planned sweep (n > 0) on `stream`. */
wsr_status run_sweep(const SweepPlan& p, int32_t n, int32_t n_tokens, void* ws, void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    unsigned* ctr = static_cast<unsigned*>(ws);
    DevMat* dtab = reinterpret_cast<DevMat*>(static_cast<char*>(ws) + wsr::SWEEP_CTR_BYTES);
    int64_t* dcost = reinterpret_cast<int64_t*>(reinterpret_cast<char*>(dtab) +
                                                ((size_t)n * sizeof(DevMat) + 255) / 256 * 256);
    /* The last tokens go in passes of the largest power of two that fits.  The table goes to the
       workspace only if some launch reads it there; the others carry it in their arguments. */
    bool upload = false;
    for (int32_t t = 0, T = p.batch; t < n_tokens && !upload; t += T) {
        while (T > n_tokens - t) T >>= 1;
        for (const Seg& g : p.segs) upload |= !wsr::sweep_table_by_value(g.count, g.total, g.fmt, T);
    }
    hipError_t e = hipSuccess;
    if (upload && (e = wsr::launch_put_table(dtab, dcost, p.tab.data(), n, ctr, s)) != hipSuccess)
        return hip_fail(e, "decode_sweep: table upload");
    for (int32_t t = 0; t < n_tokens;) {
        int32_t T = p.batch;
        while (T > n_tokens - t) T >>= 1;
        for (const Seg& g : p.segs) {
            e = wsr::launch_sweep(dtab + g.first, dcost + g.first, p.tab.data() + g.first, g.count, g.total, g.fmt,
                                  t, T, ctr, s);
            if (e != hipSuccess) return hip_fail(e, "decode_sweep: launch");
        }
        t += T;
    }
    return ok();
}

wsr_status sweep(const wsr_mat* mats, int32_t n, int32_t n_tokens, int32_t batch, void* ws,
                 size_t ws_bytes, void* stream) {
    SweepPlan p;
    wsr_status st = plan_sweep(mats, n, n_tokens, batch, ws, ws_bytes, p);
    if (st != WSR_OK || n == 0) return st;
    return run_sweep(p, n, n_tokens, ws, stream);
}

}  // namespace

extern "C" {

wsr_status wsr_decode_sweep(const wsr_mat* mats, int32_t n, int32_t n_tokens, void* ws,
                            size_t ws_bytes, void* stream) {
    return sweep(mats, n, n_tokens, 1, ws, ws_bytes, stream);
}

wsr_status wsr_decode_sweep_batched(const wsr_mat* mats, int32_t n, int32_t n_tokens, int32_t batch,
                                    void* ws, size_t ws_bytes, void* stream) {
    return sweep(mats, n, n_tokens, batch, ws, ws_bytes, stream);
}

/* wsr_decode_sweep with the library's own per-device scratch as its workspace: no allocation and
   no workspace argument.  Every argument check runs before the scratch is looked up. */
wsr_status wsr_decode_sweep_noalloc(const wsr_mat* mats, int32_t n, int32_t n_tokens, void* stream) {
    if (n < 0 || n_tokens < 1) return fail(WSR_E_ARG, "decode_sweep_noalloc: n=%d n_tokens=%d", n, n_tokens);
    if (n == 0) return ok();
    if (!mats) return fail(WSR_E_ARG, "decode_sweep_noalloc: null pointer");
    const size_t need = wsr_sweep_workspace_bytes(mats, n);
    if (need > wsr::NOALLOC_SCRATCH_BYTES)
        return fail(WSR_E_SIZE, "decode_sweep_noalloc: a table of %d matrices needs %zu bytes of scratch; "
                    "the library holds %zu (pass a workspace to wsr_decode_sweep instead)", n, need,
                    wsr::NOALLOC_SCRATCH_BYTES);
    SweepPlan p;
    wsr_status st = plan_table(mats, n, 1, n_tokens, p);
    if (st != WSR_OK) return st;
    void* ws = nullptr;
    const hipError_t e = wsr::noalloc_scratch(&ws);
    if (e != hipSuccess) return hip_fail(e, "decode_sweep_noalloc: scratch address");
    return run_sweep(p, n, n_tokens, ws, stream);
}

}  // extern "C"

/* ---- per-use copy endpoint, residency query, endpoint selection ------------------------------ */

namespace {

/* Bytes per row of a matrix as the caller stores it: weights or codes, and scales. */
void row_parts(int fmt, int64_t K, int64_t& code_row, int64_t& scale_row) {
    if (fmt == WSR_Q4) {
        code_row = K / 2;
        scale_row = (K / 32) * 2;
    } else if (fmt == WSR_I8) {
        code_row = K;
        scale_row = 2;
    } else {
        code_row = K * 2;
        scale_row = 0;
    }
}

int64_t pad256(int64_t v) { return (v + 255) / 256 * 256; }

/* Events of the staged sweep, created once per device and kept for the life of the process; a
   mutex per device serialises the enqueueing of calls that share them (a wait enqueued on an
   event refers to the record made before it, so a later call may record the events again). */
struct StageEvents {
    std::mutex mu;
    bool made = false;
    hipEvent_t start{}, copied[2]{}, consumed[2]{};
};
StageEvents g_stage_ev[64];

/* Creates the events on first use; the caller holds e.mu.  A failed creation destroys the events it
   made, so a later call starts again from nothing. */
hipError_t make_stage_events(StageEvents& e) {
    if (e.made) return hipSuccess;
    hipEvent_t* all[5] = {&e.start, &e.copied[0], &e.copied[1], &e.consumed[0], &e.consumed[1]};
    for (int i = 0; i < 5; ++i) {
        const hipError_t r = hipEventCreateWithFlags(all[i], hipEventDisableTiming);
        if (r != hipSuccess) {
            for (int j = 0; j < i; ++j) (void)hipEventDestroy(*all[j]);
            return r;
        }
    }
    e.made = true;
    return hipSuccess;
}

/* The device view of [p, p + bytes) where all of it lies in one pinned host allocation, else null
   (pageable or device memory, or an extent the runtime does not report). */
const char* pinned_view(const void* p, size_t bytes) {
    if (!p || bytes == 0) return nullptr;
    hipPointerAttribute_t a{};
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    if (a.type != hipMemoryTypeHost || a.devicePointer == nullptr) return nullptr;
    const void* start = nullptr;
    size_t size = 0;
    return pinned_extent_covers(p, a.devicePointer, bytes, &start, &size) == 1 ? static_cast<const char*>(a.devicePointer)
                                                                               : nullptr;
}

/* True for host memory the runtime has not registered (pageable). */
bool pageable(const void* p) {
    if (!p) return false;
    hipPointerAttribute_t a{};
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();                   /* do not leave the error for a later check */
        return true;
    }
    return a.type == hipMemoryTypeUnregistered;
}

/* Host threads for copies out of pageable memory: copy() splits a range into slices of at least
   4 MiB over the calling thread and up to 8 helpers and returns when all are done.  The helpers
   live for the process (detached, waiting on a condition variable); a process forked from it has
   none of them, so there, as where no helper could be started, the calling thread copies alone. */
class CopyPool {
public:
    static CopyPool& get() {
        static CopyPool* p = new CopyPool();
        return *p;
    }
    void copy(char* dst, const char* src, size_t n) {
        constexpr size_t MIN_SLICE = 4u << 20;
        const size_t parts = std::max<size_t>(1, std::min<size_t>(nthreads_ + 1, n / MIN_SLICE));
        /* a forked process takes none of the locks: one may have been held when it was forked */
        if (parts == 1 || getpid() != pid_) {
            std::memcpy(dst, src, n);
            return;
        }
        std::lock_guard<std::mutex> one(call_mu_);      /* one range at a time */
        const size_t per = (n + parts - 1) / parts;
        {
            std::lock_guard<std::mutex> l(mu_);
            jobs_.clear();
            for (size_t i = 1; i < parts; ++i) {
                const size_t a = i * per, b = std::min(n, a + per);
                if (a < b) jobs_.push_back({dst + a, src + a, b - a});
            }
            next_ = 0;
            left_ = jobs_.size();
        }
        cv_.notify_all();
        std::memcpy(dst, src, std::min(n, per));
        std::unique_lock<std::mutex> l(mu_);
        done_.wait(l, [&] { return left_ == 0; });
    }

private:
    struct Job {
        char* d;
        const char* s;
        size_t n;
    };
    CopyPool() : pid_(getpid()) {
        const unsigned hw = std::thread::hardware_concurrency();
        const unsigned want = std::max(1u, std::min(8u, hw / 2));
        unsigned made = 0;
        try {                                            /* no exception may leave the C ABI */
            for (; made < want; ++made) std::thread([this] { run(); }).detach();
        } catch (...) {
        }
        nthreads_ = made;                                /* 0: the calling thread copies alone */
    }
    void run() {
        std::unique_lock<std::mutex> l(mu_);
        for (;;) {
            cv_.wait(l, [&] { return next_ < jobs_.size(); });
            const Job j = jobs_[next_++];
            l.unlock();
            std::memcpy(j.d, j.s, j.n);
            l.lock();
            if (--left_ == 0) done_.notify_all();
        }
    }
    std::mutex call_mu_, mu_;
    std::condition_variable cv_, done_;
    std::vector<Job> jobs_;
    size_t next_ = 0, left_ = 0;
    unsigned nthreads_ = 0;
    pid_t pid_;
};

/* Pinned host halves, per device, through which the staged sweep moves pageable sources: host
   threads copy a chunk into one half while the DMA engine moves the previous chunk out of the
   other.  A copy straight from pageable memory goes through the runtime's own staging (about
   28 GB/s from a file's page-cache pages, against 57 GB/s for a pinned source).  Kept for the life
   of the process; grown (after the halves' last copies have run) when a call needs more.  The
   staged sweep's per-device mutex guards them. */
struct Bounce {
    char* half[2] = {nullptr, nullptr};
    char* view[2] = {nullptr, nullptr};                  /* their device views (null: copy with the runtime) */
    size_t bytes = 0;
    hipEvent_t out[2]{};                                 /* the last copy out of each half */
    bool pending[2] = {false, false};
    bool made = false;
};
Bounce g_bounce[64];

hipError_t bounce_ready(Bounce& b, size_t bytes) {
    hipError_t e = hipSuccess;
    if (!b.made) {
        for (int i = 0; i < 2; ++i)
            if ((e = hipEventCreateWithFlags(&b.out[i], hipEventDisableTiming)) != hipSuccess) {
                if (i == 1) (void)hipEventDestroy(b.out[0]);
                return e;
            }
        b.made = true;
    }
    if (b.bytes >= bytes) return hipSuccess;
    for (int i = 0; i < 2; ++i) {
        if (b.pending[i] && (e = hipEventSynchronize(b.out[i])) != hipSuccess) return e;
        b.pending[i] = false;
        if (b.half[i]) (void)hipHostFree(b.half[i]);
        b.half[i] = b.view[i] = nullptr;
    }
    b.bytes = 0;
    for (int i = 0; i < 2; ++i)
        if ((e = hipHostMalloc(reinterpret_cast<void**>(&b.half[i]), bytes, hipHostMallocDefault)) != hipSuccess) {
            if (i == 1) (void)hipHostFree(b.half[0]);
            b.half[0] = b.half[1] = nullptr;
            return e;
        }
    for (int i = 0; i < 2; ++i) {
        void* v = nullptr;
        if (hipHostGetDevicePointer(&v, b.half[i], 0) == hipSuccess) b.view[i] = static_cast<char*>(v);
        else (void)hipGetLastError();
    }
    b.bytes = bytes;
    return hipSuccess;
}

/* One part of a chunk into the stage on the copy stream: by the shaders from the source's device
   view where it has one and 16-byte alignment allows, else by the runtime. */
hipError_t stage_copy(char* dst, const char* src, const char* src_view, size_t bytes, hipStream_t cs) {
    if (bytes == 0) return hipSuccess;
    if (src_view && ((reinterpret_cast<uintptr_t>(src_view) | reinterpret_cast<uintptr_t>(dst) | bytes) & 15) == 0)
        return wsr::launch_copy16(src_view, dst, bytes, cs);
    return hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, cs);
}

}  // namespace

extern "C" {

wsr_status wsr_sweep_staged(const wsr_mat* mats, int32_t n, int32_t token, void* stage, size_t stage_bytes,
                            void* stream, void* copy_stream) {
    if (n < 0 || token < 0) return fail(WSR_E_ARG, "sweep_staged: n=%d token=%d", n, token);
    if (n == 0) return ok();
    if (!mats || !stage) return fail(WSR_E_ARG, "sweep_staged: null pointer");
    if (!aligned(stage, 256)) return fail(WSR_E_ALIGN, "sweep_staged: staging buffer must be 256-byte aligned");
    const int64_t half = (int64_t)(stage_bytes / 2) / 256 * 256;
    char who[64];
    for (int32_t i = 0; i < n; ++i) {
        const wsr_mat& m = mats[i];
        std::snprintf(who, sizeof who, "sweep_staged: matrix %d", i);
        wsr_status st = check_matrix(m.fmt, m.M, m.K, m.w, m.scales, m.x, m.y, who);
        if (st != WSR_OK) return st;
        if (m.flags & ~WSR_MAT_AFTER_PREVIOUS) return fail(WSR_E_ARG, "%s: unknown flags %#x", who, m.flags);
        if (m.x_tok_stride < 0 || m.y_tok_stride < 0 || m.x_tok_stride % 16 || m.y_tok_stride % 4)
            return fail(WSR_E_ALIGN, "%s: token strides must be >= 0 and multiples of 16 (x) and 4 (y)", who);
        if (!mul_fits(m.x_tok_stride, (int64_t)token + 1) || !mul_fits(m.y_tok_stride, (int64_t)token + 1))
            return fail(WSR_E_SIZE, "%s: token strides overflow", who);
        int64_t code_row, scale_row;
        row_parts(m.fmt, m.K, code_row, scale_row);
        if (m.M > 0 && code_row + scale_row > 0 && half < 256 + code_row + scale_row)
            return fail(WSR_E_SIZE, "%s: half of the staging buffer (%lld bytes) holds no row of %lld bytes", who,
                        (long long)half, (long long)(code_row + scale_row));
    }
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "sweep_staged: device");
    if (dev < 0 || dev >= 64) return fail(WSR_E_ARG, "sweep_staged: device %d", dev);
    StageEvents* ev = &g_stage_ev[dev];
    std::lock_guard<std::mutex> lock(ev->mu);       /* held from the events' creation on */
    if ((e = make_stage_events(*ev)) != hipSuccess) return hip_fail(e, "sweep_staged: events");
    hipStream_t s = static_cast<hipStream_t>(stream), cs = static_cast<hipStream_t>(copy_stream);
    char* buf[2] = {static_cast<char*>(stage), static_cast<char*>(stage) + half};
    /* The first copy waits for the work already on `stream` (an earlier reader of the buffer). */
    if ((e = hipEventRecord(ev->start, s)) != hipSuccess || (e = hipStreamWaitEvent(cs, ev->start, 0)) != hipSuccess)
        return hip_fail(e, "sweep_staged: ordering");
    int64_t k = 0, kb = 0;                           /* chunks; chunks through the bounce halves */
    Bounce* bo = nullptr;
    for (int32_t i = 0; i < n; ++i) {
        const wsr_mat& m = mats[i];
        if (m.M == 0) continue;
        int64_t code_row, scale_row;
        row_parts(m.fmt, m.K, code_row, scale_row);
        /* a pageable part goes through a pinned bounce half, the others straight to the stage; the
           shaders copy what is in pinned host pages (the copy engines halved that rate in some
           processes), the runtime the rest */
        const bool pw = pageable(m.w), ps = scale_row > 0 && pageable(m.scales);
        const char* wview = pw ? nullptr : pinned_view(m.w, (size_t)(m.M * code_row));
        const char* sview = ps || scale_row == 0 ? nullptr : pinned_view(m.scales, (size_t)(m.M * scale_row));
        if ((pw || ps) && !bo) {
            bo = &g_bounce[dev];
            if ((e = bounce_ready(*bo, (size_t)half)) != hipSuccess) return hip_fail(e, "sweep_staged: pinned bounce");
        }
        const int64_t per = code_row + scale_row > 0 ? (half - 256) / (code_row + scale_row) : m.M;
        const char* x = static_cast<const char*>(m.x) + (int64_t)token * m.x_tok_stride;
        char* y = reinterpret_cast<char*>(m.y) + (int64_t)token * m.y_tok_stride;
        for (int64_t r0 = 0; r0 < m.M; r0 += per, ++k) {
            const int64_t rows = std::min<int64_t>(per, m.M - r0);
            const int b = (int)(k & 1);
            const int64_t soff = pad256(rows * code_row);
            /* Buffer b is free once the GEMV of the chunk two back has run. */
            if (k >= 2 && (e = hipStreamWaitEvent(cs, ev->consumed[b], 0)) != hipSuccess)
                return hip_fail(e, "sweep_staged: wait");
            const char* wsrc = static_cast<const char*>(m.w) + r0 * code_row;
            const char* ssrc = scale_row > 0 ? static_cast<const char*>(m.scales) + r0 * scale_row : nullptr;
            const char* wdev = wview ? wview + r0 * code_row : nullptr;       /* device views, if pinned */
            const char* sdev = sview ? sview + r0 * scale_row : nullptr;
            if (pw || ps) {
                /* the host fills bounce half bb once its last copy out has run */
                const int bb = (int)(kb++ & 1);
                if (bo->pending[bb] && (e = hipEventSynchronize(bo->out[bb])) != hipSuccess)
                    return hip_fail(e, "sweep_staged: host wait");
                if (pw && rows * code_row > 0) {
                    CopyPool::get().copy(bo->half[bb], wsrc, (size_t)(rows * code_row));
                    wsrc = bo->half[bb];
                    wdev = bo->view[bb];
                }
                if (ps) {
                    CopyPool::get().copy(bo->half[bb] + soff, ssrc, (size_t)(rows * scale_row));
                    ssrc = bo->half[bb] + soff;
                    sdev = bo->view[bb] ? bo->view[bb] + soff : nullptr;
                }
            }
            if ((e = stage_copy(buf[b], wsrc, wdev, (size_t)(rows * code_row), cs)) != hipSuccess)
                return hip_fail(e, "sweep_staged: copy");
            if (scale_row > 0 && (e = stage_copy(buf[b] + soff, ssrc, sdev, (size_t)(rows * scale_row), cs)) != hipSuccess)
                return hip_fail(e, "sweep_staged: copy");
            if (pw || ps) {
                const int bb = (int)((kb - 1) & 1);
                if ((e = hipEventRecord(bo->out[bb], cs)) != hipSuccess) return hip_fail(e, "sweep_staged: ordering");
                bo->pending[bb] = true;
            }
            if ((e = hipEventRecord(ev->copied[b], cs)) != hipSuccess || (e = hipStreamWaitEvent(s, ev->copied[b], 0)) != hipSuccess)
                return hip_fail(e, "sweep_staged: ordering");
            const DevMat d = make_devmat(m.fmt, rows, m.K, buf[b], scale_row > 0 ? buf[b] + soff : nullptr, x,
                                         reinterpret_cast<float*>(y + r0 * 4));
            if ((e = wsr::launch_gemv(d, s)) != hipSuccess) return hip_fail(e, "sweep_staged: launch");
            if ((e = hipEventRecord(ev->consumed[b], s)) != hipSuccess) return hip_fail(e, "sweep_staged: ordering");
        }
    }
    return ok();
}

wsr_status wsr_host_resident_pages(const void* host, size_t bytes, size_t* resident_pages, size_t* total_pages) {
    if (!host || !resident_pages || !total_pages) return fail(WSR_E_ARG, "host_resident_pages: null pointer");
    const long pg = sysconf(_SC_PAGESIZE);
    const uintptr_t a = reinterpret_cast<uintptr_t>(host) / pg * pg;
    const uintptr_t end = (reinterpret_cast<uintptr_t>(host) + bytes + pg - 1) / pg * pg;
    const size_t np = (end - a) / pg;
    std::vector<unsigned char> v(np ? np : 1);
    if (np && mincore(reinterpret_cast<void*>(a), end - a, v.data()) != 0)
        return fail(WSR_E_ARG, "host_resident_pages: range is not mapped");
    size_t r = 0;
    for (size_t i = 0; i < np; ++i) r += v[i] & 1;
    *resident_pages = r;
    *total_pages = np;
    return ok();
}

wsr_status wsr_select_endpoint(const wsr_endpoint_probe* p, double theta, int32_t* choice, double* times_ms) {
    if (!p || !choice) return fail(WSR_E_ARG, "select_endpoint: null pointer");
    if (!(theta >= 0.0) || !(p->w_bytes > 0.0)) return fail(WSR_E_ARG, "select_endpoint: theta and W must be >= 0 and > 0");
    if (p->excluded & ~((1u << WSR_EP_MAP) | (1u << WSR_EP_RESIDENT) | (1u << WSR_EP_COPY)))
        return fail(WSR_E_ARG, "select_endpoint: unknown endpoint in the exclusion mask %#x", p->excluded);
    const int eps[3] = {WSR_EP_MAP, WSR_EP_RESIDENT, WSR_EP_COPY};
    double t[3];
    for (int j = 0; j < 3; ++j) {
        const double b = p->rate[j];
        t[j] = b > 0.0 ? p->w_bytes / b * 1e3 : -1.0;
        if (times_ms) times_ms[j] = t[j];
    }
    /* Storage-bound stop: the mapped set is not resident after prefaulting. */
    if (!p->mapped_resident) {
        *choice = WSR_EP_STORAGE_BOUND;
        return ok();
    }
    bool live[3];
    for (int j = 0; j < 3; ++j) live[j] = t[j] > 0.0 && !(p->excluded & (1u << eps[j]));
    if (!p->resident_ok) live[1] = false;     /* allocation failed, or it evicted the mapping */
    int best = -1;
    for (int j = 0; j < 3; ++j)
        if (live[j] && (best < 0 || t[j] < t[best])) best = j;
    if (best < 0) {
        *choice = WSR_EP_NONE;
        return ok();
    }
    /* Tie band: mapping wins when its time is within theta of the fastest survivor. */
    if (live[0] && t[0] - t[best] <= theta * t[best]) best = 0;
    *choice = eps[best];
    return ok();
}

}  // extern "C"

/* ---- matrix-core sweep ---------------------------------------------------------------------------- */

extern "C" wsr_status wsr_decode_sweep_mma(const wsr_mat* mats, int32_t n, int32_t n_tokens, void* ws, size_t ws_bytes,
                                           void* stream) {
    SweepPlan p;
    wsr_status st = plan_sweep(mats, n, n_tokens, n_tokens > 1 ? 16 : 1, ws, ws_bytes, p);
    if (st != WSR_OK || n == 0) return st;
    for (int32_t i = 0; i < n; ++i)       /* 64 rows and 16 tokens within 32-bit lane offsets */
        if (p.tab[i].nc * 16 > (int64_t{1} << 25) || p.tab[i].x_stride > (int64_t{1} << 27))
            return fail(WSR_E_SIZE, "decode_sweep_mma: matrix %d: rows above 32 MiB or x_tok_stride above 128 MiB", i);
    hipStream_t s = static_cast<hipStream_t>(stream);
    unsigned* ctr = static_cast<unsigned*>(ws);
    DevMat* dtab = reinterpret_cast<DevMat*>(static_cast<char*>(ws) + wsr::SWEEP_CTR_BYTES);
    int64_t* dcost = reinterpret_cast<int64_t*>(reinterpret_cast<char*>(dtab) +
                                                ((size_t)n * sizeof(DevMat) + 255) / 256 * 256);
    /* the matrix-core launches read the table from the workspace; a single-token pass may carry it
       in its arguments */
    bool upload = false;
    for (int32_t t = 0; t < n_tokens && !upload; t += 16)
        for (const Seg& g : p.segs)
            upload |= std::min<int32_t>(16, n_tokens - t) > 1 || !wsr::sweep_table_by_value(g.count, g.total, g.fmt, 1);
    hipError_t e = hipSuccess;
    if (upload && (e = wsr::launch_put_table(dtab, dcost, p.tab.data(), n, ctr, s)) != hipSuccess)
        return hip_fail(e, "decode_sweep_mma: table upload");
    /* per segment: the largest row group of 64 and of 128 rows, of the tail's rows, and the longest row */
    std::vector<int64_t> max_g4(p.segs.size(), 0), max_g8(p.segs.size(), 0), max_tail(p.segs.size(), 0),
        max_row(p.segs.size(), 0);
    for (size_t i = 0; i < p.segs.size(); ++i)
        for (int m = p.segs[i].first; m < p.segs[i].first + p.segs[i].count; ++m) {
            const int64_t rb = p.tab[m].row_bytes, M = p.tab[m].M;
            max_g4[i] = std::max(max_g4[i], rb * std::min<int64_t>(M, 64));
            max_g8[i] = std::max(max_g8[i], rb * std::min<int64_t>(M, 128));
            max_tail[i] = std::max(max_tail[i], rb * std::min(M, wsr::mma_tail_rows()));
            max_row[i] = std::max(max_row[i], p.tab[m].nc * 16);
        }
    std::vector<int> mma_fmt(p.segs.size());
    for (size_t i = 0; i < p.segs.size(); ++i) {
        const Seg& g = p.segs[i];
        bool whole = g.fmt == WSR_Q4;
        for (int m = g.first; whole && m < g.first + g.count; ++m)
            whole = p.tab[m].nc % 8 == 0 && (reinterpret_cast<uintptr_t>(p.tab[m].s) & 15) == 0;
        mma_fmt[i] = whole ? wsr::FMT_Q4_WHOLE : g.fmt;
    }
    for (int32_t t = 0; t < n_tokens; t += 16) {
        const int ntok = std::min<int32_t>(16, n_tokens - t);
        for (size_t i = 0; i < p.segs.size(); ++i) {
            const Seg& g = p.segs[i];
            /* a pass of one token would fill 16 token slots of every matrix instruction for one; the
               vector-ALU loop serves it instead (8B q4: 1.6k tok/s against 1.0k) */
            const int tiles = wsr::mma_tiles(mma_fmt[i], ntok, max_row[i]);
            e = ntok == 1 ? wsr::launch_sweep(dtab + g.first, dcost + g.first, p.tab.data() + g.first, g.count, g.total,
                                              g.fmt, t, 1, ctr, s)
                          : wsr::launch_sweep_mma(dtab + g.first, dcost + g.first, g.count, g.total, tiles,
                                                  tiles == 8 ? max_g8[i] : max_g4[i], max_tail[i], mma_fmt[i], t,
                                                  ntok, s);
            if (e != hipSuccess) return hip_fail(e, "decode_sweep_mma: launch");
        }
    }
    return ok();
}

/* ---- a decode pass ordered against another stream (execution contract C3, Sec. 4.3) ----------- */

namespace {

struct OrderEvents {
    std::mutex mu;
    bool made = false;
    hipEvent_t before{}, after{};
};
OrderEvents g_order_ev[64];

}  // namespace

extern "C" {

wsr_status wsr_decode_sweep_ordered(const wsr_mat* mats, int32_t n, int32_t n_tokens, void* ws, size_t ws_bytes,
                                    void* framework_stream, void* own_stream, int32_t mode) {
    if (mode < WSR_ORDER_STREAM || mode > WSR_ORDER_DRAIN)
        return fail(WSR_E_ARG, "decode_sweep_ordered: unknown mode %d", mode);
    if (mode == WSR_ORDER_STREAM) return sweep(mats, n, n_tokens, 1, ws, ws_bytes, framework_stream);
    SweepPlan p;
    wsr_status st = plan_sweep(mats, n, n_tokens, 1, ws, ws_bytes, p);
    if (st != WSR_OK || n == 0) return st;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "decode_sweep_ordered: device");
    if (dev < 0 || dev >= 64) return fail(WSR_E_ARG, "decode_sweep_ordered: device %d", dev);
    OrderEvents& ev = g_order_ev[dev];
    std::lock_guard<std::mutex> lock(ev.mu);
    if (!ev.made) {
        if ((e = hipEventCreateWithFlags(&ev.before, hipEventDisableTiming)) != hipSuccess)
            return hip_fail(e, "decode_sweep_ordered: events");
        if ((e = hipEventCreateWithFlags(&ev.after, hipEventDisableTiming)) != hipSuccess) {
            (void)hipEventDestroy(ev.before);
            return hip_fail(e, "decode_sweep_ordered: events");
        }
        ev.made = true;
    }
    hipStream_t fs = static_cast<hipStream_t>(framework_stream), os = static_cast<hipStream_t>(own_stream);
    /* Before the pass: the framework's work so far must be complete. */
    if (mode == WSR_ORDER_DRAIN) {
        if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "decode_sweep_ordered: drain");
    } else {
        if ((e = hipEventRecord(ev.before, fs)) != hipSuccess) return hip_fail(e, "decode_sweep_ordered: record");
        if (mode == WSR_ORDER_EVENT)
            e = hipStreamWaitEvent(os, ev.before, 0);
        else
            e = hipEventSynchronize(ev.before);       /* the host observes the signal */
        if (e != hipSuccess) return hip_fail(e, "decode_sweep_ordered: wait");
    }
    st = run_sweep(p, n, n_tokens, ws, own_stream);
    if (st != WSR_OK) return st;
    /* After the pass: the framework's later work waits for it on the GPU. */
    if ((e = hipEventRecord(ev.after, os)) != hipSuccess || (e = hipStreamWaitEvent(fs, ev.after, 0)) != hipSuccess)
        return hip_fail(e, "decode_sweep_ordered: order after");
    return ok();
}

}  // extern "C"
