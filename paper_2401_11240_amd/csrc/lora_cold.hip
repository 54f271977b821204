// Cold start (Section 2.3 C1, Section 4.1, Section 4.2): stream-ordered
// signals into pinned host memory, the sync-free hand-off of x to the host,
// the asynchronous adapter load, and the merge of a CPU-computed delta.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cstdint>
#include <string>

#include "lora.h"
#include "lora_coldstart.h"
#include "lora_device.h"
#include "lora_internal.h"

namespace lora {
int set_error(int code, const std::string& msg);
}

using namespace lora;

namespace {

// One wave: the flag store, released at system scope (the CPU reads it).  It
// runs after the work queued before it on the stream has completed.
__global__ void __launch_bounds__(64) lora_signal_kernel(uint32_t* flag, uint32_t value) {
    if (threadIdx.x == 0) __hip_atomic_store(flag, value, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// y = round(y + delta), four consecutive elements per thread.
constexpr int kAddThreads = 256;

template <class Fmt>
__global__ void __launch_bounds__(kAddThreads) lora_add_delta_kernel(const float* delta, int64_t ld_delta, uint16_t* y,
                                                                     int64_t ldy, int32_t n_rows, int32_t quads) {
    const int64_t i = (int64_t)blockIdx.x * kAddThreads + threadIdx.x;
    const int64_t t = i / quads;
    if (t >= n_rows) return;
    const int q = (int)(i - t * quads);
    const float4 d = *(const float4*)(delta + t * ld_delta + 4 * q);
    uint2* yp = (uint2*)(y + t * ldy + 4 * q);
    const uint2 v = *yp;
    const float y0 = Fmt::to_f32(v.x & 0xffffu) + d.x, y1 = Fmt::to_f32(v.x >> 16) + d.y;
    const float y2 = Fmt::to_f32(v.y & 0xffffu) + d.z, y3 = Fmt::to_f32(v.y >> 16) + d.w;
    *yp = uint2{Fmt::pack2(y0, y1), Fmt::pack2(y2, y3)};
}

// The device a stream belongs to current for the launch.
struct StreamDevice {
    int prev = -1;
    bool ok = false;
    explicit StreamDevice(hipStream_t s) {
        int dev = -1;
        if (hipGetDevice(&prev) != hipSuccess) return;
        if (s) {
            if (hipStreamGetDevice(s, &dev) != hipSuccess) return;
        } else {
            dev = prev;
        }
        ok = dev == prev || hipSetDevice(dev) == hipSuccess;
    }
    ~StreamDevice() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

int enqueue_signal(uint32_t* flag, uint32_t value, hipStream_t s) {
    hipLaunchKernelGGL(lora_signal_kernel, dim3(1), dim3(64), 0, s, flag, value);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(LORA_E_HIP, std::string("signal kernel: ") + hipGetErrorString(e));
    return LORA_OK;
}

bool reached(uint32_t flag, uint32_t value) { return (int32_t)(flag - value) >= 0; }

}  // namespace

extern "C" {

int lora_host_alloc(size_t bytes, void** out) {
    if (!out) return set_error(LORA_E_ARG, "lora_host_alloc: out is NULL");
    *out = nullptr;
    const hipError_t e = hipHostMalloc(out, bytes ? bytes : 1, hipHostMallocCoherent | hipHostMallocPortable);
    if (e != hipSuccess) {
        *out = nullptr;
        return set_error(LORA_E_NOMEM, std::string("lora_host_alloc: ") + hipGetErrorString(e));
    }
    return LORA_OK;
}

int lora_host_free(void* p) {
    if (!p) return LORA_OK;
    const hipError_t e = hipHostFree(p);
    if (e != hipSuccess) return set_error(LORA_E_HIP, std::string("lora_host_free: ") + hipGetErrorString(e));
    return LORA_OK;
}

int lora_signal(uint32_t* host_flag, uint32_t value, void* stream) {
    if (!host_flag) return set_error(LORA_E_ARG, "lora_signal: host_flag is NULL");
    hipStream_t s = (hipStream_t)stream;
    StreamDevice g(s);
    if (!g.ok) return set_error(LORA_E_HIP, "lora_signal: cannot select the stream's device");
    return enqueue_signal(host_flag, value, s);
}

int lora_handoff_x(const void* x, int64_t ldx, int32_t n_rows, int32_t h, void* host_x, int64_t ld_host,
                   uint32_t* host_flag, uint32_t value, void* stream) {
    if (!host_flag) return set_error(LORA_E_ARG, "lora_handoff_x: host_flag is NULL");
    if (n_rows < 0 || h < 1) return set_error(LORA_E_ARG, "lora_handoff_x: needs n_rows >= 0 and h >= 1");
    if (n_rows > 0 && (!x || !host_x)) return set_error(LORA_E_ARG, "lora_handoff_x: x or host_x is NULL");
    if (ldx < h || ld_host < h) return set_error(LORA_E_SHAPE, "lora_handoff_x: ldx and ld_host must be >= h");
    hipStream_t s = (hipStream_t)stream;
    StreamDevice g(s);
    if (!g.ok) return set_error(LORA_E_HIP, "lora_handoff_x: cannot select the stream's device");
    if (n_rows > 0) {
        const hipError_t e = hipMemcpy2DAsync(host_x, (size_t)ld_host * 2, x, (size_t)ldx * 2, (size_t)h * 2,
                                              (size_t)n_rows, hipMemcpyDeviceToHost, s);
        if (e != hipSuccess)
            return set_error(LORA_E_HIP, std::string("lora_handoff_x copy: ") + hipGetErrorString(e));
    }
    return enqueue_signal(host_flag, value, s);
}

int lora_adapter_load_async(void* dst_dev, const void* src_host, size_t bytes, uint32_t* host_flag, uint32_t value,
                            void* stream) {
    if (!host_flag) return set_error(LORA_E_ARG, "lora_adapter_load_async: host_flag is NULL");
    if (bytes > 0 && (!dst_dev || !src_host))
        return set_error(LORA_E_ARG, "lora_adapter_load_async: dst_dev or src_host is NULL");
    hipStream_t s = (hipStream_t)stream;
    StreamDevice g(s);
    if (!g.ok) return set_error(LORA_E_HIP, "lora_adapter_load_async: cannot select the stream's device");
    if (bytes > 0) {
        const hipError_t e = hipMemcpyAsync(dst_dev, src_host, bytes, hipMemcpyHostToDevice, s);
        if (e != hipSuccess)
            return set_error(LORA_E_HIP, std::string("lora_adapter_load_async copy: ") + hipGetErrorString(e));
    }
    return enqueue_signal(host_flag, value, s);
}

int lora_flag_test(const uint32_t* host_flag, uint32_t value) {
    if (!host_flag) return -1;
    return reached(__atomic_load_n(host_flag, __ATOMIC_ACQUIRE), value) ? 1 : 0;
}

int lora_flag_wait(const uint32_t* host_flag, uint32_t value, int64_t timeout_ns) {
    if (!host_flag) return set_error(LORA_E_ARG, "lora_flag_wait: host_flag is NULL");
    const auto t0 = std::chrono::steady_clock::now();
    for (uint64_t it = 0;; ++it) {
        if (reached(__atomic_load_n(host_flag, __ATOMIC_ACQUIRE), value)) return LORA_OK;
        if (timeout_ns >= 0 && (it & 255) == 0) {
            const auto dt = std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - t0);
            if (dt.count() > timeout_ns)
                return set_error(LORA_E_SYNC, "lora_flag_wait: timed out waiting for " + std::to_string(value));
        }
        __builtin_ia32_pause();
    }
}

int lora_add_delta(const float* delta, int64_t ld_delta, void* y, int64_t ldy, int32_t n_rows, int32_t h_out,
                   int32_t dtype, void* stream) {
    if (n_rows < 0 || h_out < 1) return set_error(LORA_E_ARG, "lora_add_delta: needs n_rows >= 0 and h_out >= 1");
    if (dtype != LORA_F16 && dtype != LORA_BF16) return set_error(LORA_E_ARG, "lora_add_delta: bad dtype");
    if (n_rows == 0) return LORA_OK;
    if (!delta || !y) return set_error(LORA_E_ARG, "lora_add_delta: delta or y is NULL");
    if (h_out % 4 || ldy % 4 || ld_delta % 4 || ldy < h_out || ld_delta < h_out)
        return set_error(LORA_E_SHAPE, "lora_add_delta: h_out, ldy and ld_delta must be multiples of 4, ld >= h_out");
    if (((uintptr_t)delta & 15) || ((uintptr_t)y & 7))
        return set_error(LORA_E_ALIGN, "lora_add_delta: delta must be 16-byte and y 8-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    StreamDevice g(s);
    if (!g.ok) return set_error(LORA_E_HIP, "lora_add_delta: cannot select the stream's device");
    const int32_t quads = h_out / 4;
    const int64_t n = (int64_t)n_rows * quads;
    const int64_t blocks = (n + kAddThreads - 1) / kAddThreads;
    if (blocks > 0x7fffffff) return set_error(LORA_E_SHAPE, "lora_add_delta: too many rows");
    if (dtype == LORA_F16)
        hipLaunchKernelGGL(lora_add_delta_kernel<FmtF16>, dim3((uint32_t)blocks), dim3(kAddThreads), 0, s, delta,
                           ld_delta, (uint16_t*)y, ldy, n_rows, quads);
    else
        hipLaunchKernelGGL(lora_add_delta_kernel<FmtBF16>, dim3((uint32_t)blocks), dim3(kAddThreads), 0, s, delta,
                           ld_delta, (uint16_t*)y, ldy, n_rows, quads);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(LORA_E_HIP, std::string("lora_add_delta: ") + hipGetErrorString(e));
    return LORA_OK;
}

}  // extern "C"
