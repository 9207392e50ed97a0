// Host-resident records: the outer-time path (dt_pipeline_* and dt_*classify_host in
// include/dtree.h).
//
// Section 4.2 of the paper measures each GPU function from the host: allocate, copy the
// records in, run the kernel, copy the labels out, free, all in series; Section 4.3 finds
// those copies dominate and points at pinned buffers and copies overlapped with compute.
// A pipeline keeps `n_slots` chunk buffers on the device, each with its own stream (default
// priority) and pinned bounce buffers.  Chunk c goes to slot c % n_slots: copy in, classify
// and copy out are queued on that slot's stream, so while one chunk is classified the next
// is already crossing PCIe and the previous one's labels are coming back.  Before a slot is
// reused its previous chunk is retired (its last event waited for, its labels moved to the
// caller's buffer if they came through a bounce buffer).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstring>
#include <functional>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "dtree.h"
#include "library.hpp"

namespace {

using dtree::set_error;
using dtree::set_hip_error;

constexpr int kDefaultSlots = 3;
constexpr int kMaxSlots = 8;
constexpr int kDefaultHostThreads = 4;
constexpr int kMaxHostThreads = 16;
constexpr int64_t kMinBytesPerThread = int64_t(1) << 20;
constexpr int64_t kDefaultChunkBytes = int64_t(32) << 20;
constexpr int32_t kMaxFeatures = 256;
constexpr int64_t kMaxRows = int64_t(1) << 37;

enum { kEvIn = 0, kEvKernel, kEvOut, kEvDone, kEvents };

struct Slot {
    hipStream_t stream = nullptr;
    hipEvent_t ev[kEvents] = {};
    char *d_x = nullptr;       // chunk_rows x n_features x 4 bytes (any record type fits)
    void *d_out = nullptr;     // chunk_rows x 4 bytes
    char *h_x = nullptr;       // pinned bounce buffer for records
    void *h_out = nullptr;     // pinned bounce buffer for labels
    bool busy = false;         // a chunk is queued and not yet retired
    int64_t row0 = 0, rows = 0;
};

// Classify `rows` device-resident records (dense rows of n_features elements) on `stream`.
using ClassifyFn = std::function<dt_status(const void *, int64_t, void *, hipStream_t)>;

bool is_page_locked(const void *p) {
    if (!p) return false;
    hipPointerAttribute_t attr{};
    const hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();   // pageable memory is not an error here
        return false;
    }
    return attr.type == hipMemoryTypeHost;
}

// Copy `rows` records of row_bytes bytes (source row stride ld_bytes) into the dense
// buffer dst, split over up to `threads` host threads (the calling one included).
void pack_rows(char *dst, const char *src, int64_t rows, int64_t ld_bytes, int64_t row_bytes,
               int threads) {
    const auto work = [=](int64_t r0, int64_t r1) {
        if (r0 >= r1) return;
        if (ld_bytes == row_bytes) {
            std::memcpy(dst + r0 * row_bytes, src + r0 * ld_bytes, size_t((r1 - r0) * row_bytes));
        } else {
            for (int64_t r = r0; r < r1; ++r)
                std::memcpy(dst + r * row_bytes, src + r * ld_bytes, size_t(row_bytes));
        }
    };
    const int64_t bytes = rows * row_bytes;
    const int t = int(std::max<int64_t>(1, std::min<int64_t>(threads, bytes / kMinBytesPerThread)));
    const int64_t per = (rows + t - 1) / t;
    std::vector<std::thread> pool;
    int started = 1;
    try {
        pool.reserve(size_t(t - 1));
        for (; started < t; ++started)
            pool.emplace_back(work, started * per, std::min(rows, (started + 1) * per));
    } catch (...) {
        // no more threads: the calling thread copies the slices that did not start
    }
    work(0, std::min(rows, per));
    for (int k = started; k < t; ++k) work(k * per, std::min(rows, (k + 1) * per));
    for (std::thread &th : pool) th.join();
}

double elapsed_us(hipEvent_t a, hipEvent_t b) {
    float ms = 0.f;
    return hipEventElapsedTime(&ms, a, b) == hipSuccess ? double(ms) * 1e3 : 0.0;
}

}  // namespace

struct dt_pipeline {
    int device = -1;
    int32_t n_features = 0;
    int64_t chunk_rows = 0;
    int host_threads = 1;
    bool serial = false;
    std::vector<Slot> slots;
};

namespace {

void release(dt_pipeline *p) {
    for (Slot &s : p->slots) {
        if (s.stream) (void)hipStreamSynchronize(s.stream);
        for (hipEvent_t &e : s.ev)
            if (e) (void)hipEventDestroy(e);
        if (s.stream) (void)hipStreamDestroy(s.stream);
        if (s.d_x) (void)hipFree(s.d_x);
        if (s.d_out) (void)hipFree(s.d_out);
        if (s.h_x) (void)hipHostFree(s.h_x);
        if (s.h_out) (void)hipHostFree(s.h_out);
    }
    p->slots.clear();
}

dt_status create_impl(int32_t n_features, const dt_pipeline_options *opt, dt_pipeline **out) {
    if (!out) return set_error(DT_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (n_features < 1 || n_features > kMaxFeatures)
        return set_error(DT_ERR_INVALID_ARG, "n_features must be 1..256");
    dt_pipeline_options o{};
    if (opt) o = *opt;
    if (o.chunk_rows < 0) return set_error(DT_ERR_INVALID_ARG, "chunk_rows must be >= 0");
    if (o.n_slots < 0 || o.n_slots > kMaxSlots)
        return set_error(DT_ERR_INVALID_ARG, "n_slots must be 0 (auto) or 1..8");
    if (o.serial != 0 && o.serial != 1) return set_error(DT_ERR_INVALID_ARG, "serial must be 0 or 1");
    if (o.host_threads < 0 || o.host_threads > kMaxHostThreads)
        return set_error(DT_ERR_INVALID_ARG, "host_threads must be 0 (auto) or 1..16");

    dt_pipeline *p = new (std::nothrow) dt_pipeline();
    if (!p) return set_error(DT_ERR_NO_MEMORY, "host allocation failed");
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) {
        delete p;
        return set_hip_error(e, "hipGetDevice");
    }
    p->n_features = n_features;
    p->serial = o.serial == 1;
    p->host_threads = o.host_threads ? o.host_threads : kDefaultHostThreads;
    const int64_t row_bytes = int64_t(n_features) * 4;
    int64_t rows = o.chunk_rows ? o.chunk_rows : std::max<int64_t>(1, kDefaultChunkBytes / row_bytes);
    rows = std::min(kMaxRows, (rows + 63) / 64 * 64);
    p->chunk_rows = rows;
    const int n_slots = p->serial ? 1 : (o.n_slots ? o.n_slots : kDefaultSlots);
    p->slots.resize(size_t(n_slots));
    for (Slot &s : p->slots) {
        e = hipStreamCreateWithFlags(&s.stream, hipStreamNonBlocking);
        for (int k = 0; e == hipSuccess && k < kEvents; ++k) e = hipEventCreate(&s.ev[k]);
        if (e != hipSuccess) {
            release(p);
            delete p;
            return set_hip_error(e, "stream or event creation");
        }
        if (p->serial) continue;   // buffers are allocated per call
        const size_t xb = size_t(rows * row_bytes), ob = size_t(rows) * 4;
        if (hipMalloc(reinterpret_cast<void **>(&s.d_x), xb) != hipSuccess ||
            hipMalloc(&s.d_out, ob) != hipSuccess ||
            hipHostMalloc(reinterpret_cast<void **>(&s.h_x), xb, hipHostMallocDefault) != hipSuccess ||
            hipHostMalloc(&s.h_out, ob, hipHostMallocDefault) != hipSuccess) {
            (void)hipGetLastError();
            release(p);
            delete p;
            return set_error(DT_ERR_NO_MEMORY, "pipeline buffer allocation failed");
        }
    }
    *out = p;
    return DT_OK;
}

// Wait for a slot's chunk, add its event times, deliver bounced labels.
dt_status retire(Slot &s, bool out_pinned, unsigned char *h_out, int esize,
                 dt_pipeline_stats *st) {
    if (!s.busy) return DT_OK;
    s.busy = false;
    const hipError_t e = hipEventSynchronize(s.ev[kEvDone]);
    if (e != hipSuccess) return set_hip_error(e, "hipEventSynchronize");
    st->h2d_us += elapsed_us(s.ev[kEvIn], s.ev[kEvKernel]);
    st->kernel_us += elapsed_us(s.ev[kEvKernel], s.ev[kEvOut]);
    st->d2h_us += elapsed_us(s.ev[kEvOut], s.ev[kEvDone]);
    if (!out_pinned)
        std::memcpy(h_out + s.row0 * esize, s.h_out, size_t(s.rows * esize));
    return DT_OK;
}

// Leave nothing of a failed call running.
void drain(dt_pipeline *p) {
    for (Slot &s : p->slots) {
        (void)hipStreamSynchronize(s.stream);
        s.busy = false;
    }
    (void)hipGetLastError();
}

dt_status run_chunked(dt_pipeline *p, const ClassifyFn &classify, const char *h_x, int xsize,
                      int64_t n, int64_t ld, unsigned char *h_out, int esize,
                      dt_pipeline_stats *st) {
    const int32_t F = p->n_features;
    const size_t row_bytes = size_t(F) * size_t(xsize);
    const int64_t ld_bytes = ld * xsize;
    const bool in_pinned = is_page_locked(h_x);
    const bool out_pinned = is_page_locked(h_out);
    st->input_pinned = in_pinned ? 1 : 0;
    st->output_pinned = out_pinned ? 1 : 0;
    const int64_t n_chunks = (n + p->chunk_rows - 1) / p->chunk_rows;
    st->chunks = n_chunks;
    const int n_slots = int(p->slots.size());
    for (int64_t c = 0; c < n_chunks; ++c) {
        Slot &s = p->slots[size_t(c % n_slots)];
        dt_status rs = retire(s, out_pinned, h_out, esize, st);
        if (rs != DT_OK) {
            drain(p);
            return rs;
        }
        s.row0 = c * p->chunk_rows;
        s.rows = std::min(p->chunk_rows, n - s.row0);
        const char *src = h_x + s.row0 * ld_bytes;
        int64_t src_ld = ld_bytes;
        if (!in_pinned) {   // pack into the slot's pinned buffer (the slot is idle now)
            pack_rows(s.h_x, src, s.rows, ld_bytes, int64_t(row_bytes), p->host_threads);
            src = s.h_x;
            src_ld = int64_t(row_bytes);
        }
        hipError_t e = hipEventRecord(s.ev[kEvIn], s.stream);
        if (e == hipSuccess) {
            if (src_ld == int64_t(row_bytes))
                e = hipMemcpyAsync(s.d_x, src, size_t(s.rows) * row_bytes, hipMemcpyHostToDevice,
                                   s.stream);
            else
                e = hipMemcpy2DAsync(s.d_x, row_bytes, src, size_t(src_ld), row_bytes,
                                     size_t(s.rows), hipMemcpyHostToDevice, s.stream);
        }
        if (e == hipSuccess) e = hipEventRecord(s.ev[kEvKernel], s.stream);
        if (e != hipSuccess) {
            drain(p);
            return set_hip_error(e, "record copy");
        }
        rs = classify(s.d_x, s.rows, s.d_out, s.stream);
        if (rs != DT_OK) {
            drain(p);
            return rs;
        }
        void *dst = out_pinned ? static_cast<void *>(h_out + s.row0 * esize) : s.h_out;
        e = hipEventRecord(s.ev[kEvOut], s.stream);
        if (e == hipSuccess)
            e = hipMemcpyAsync(dst, s.d_out, size_t(s.rows * esize), hipMemcpyDeviceToHost,
                               s.stream);
        if (e == hipSuccess) e = hipEventRecord(s.ev[kEvDone], s.stream);
        if (e != hipSuccess) {
            drain(p);
            return set_hip_error(e, "label copy");
        }
        s.busy = true;
    }
    for (Slot &s : p->slots) {
        const dt_status rs = retire(s, out_pinned, h_out, esize, st);
        if (rs != DT_OK) {
            drain(p);
            return rs;
        }
    }
    return DT_OK;
}

// Section 4.2's scheme: device buffers for all n records allocated and freed per call,
// blocking copies, the kernel in between.
dt_status run_serial(dt_pipeline *p, const ClassifyFn &classify, const char *h_x, int xsize,
                     int64_t n, int64_t ld, unsigned char *h_out, int esize,
                     dt_pipeline_stats *st) {
    using clock = std::chrono::steady_clock;
    Slot &s = p->slots[0];
    const int32_t F = p->n_features;
    const size_t row_bytes = size_t(F) * size_t(xsize);
    st->input_pinned = is_page_locked(h_x) ? 1 : 0;
    st->output_pinned = is_page_locked(h_out) ? 1 : 0;
    st->chunks = 1;
    char *d_x = nullptr;
    void *d_out = nullptr;
    if (hipMalloc(reinterpret_cast<void **>(&d_x), size_t(n) * row_bytes) != hipSuccess ||
        hipMalloc(&d_out, size_t(n * esize)) != hipSuccess) {
        (void)hipGetLastError();
        if (d_x) (void)hipFree(d_x);
        return set_error(DT_ERR_NO_MEMORY, "hipMalloc of the record buffers failed");
    }
    dt_status rs = DT_OK;
    auto t0 = clock::now();
    hipError_t e = ld == F ? hipMemcpy(d_x, h_x, size_t(n) * row_bytes, hipMemcpyHostToDevice)
                           : hipMemcpy2D(d_x, row_bytes, h_x, size_t(ld) * size_t(xsize),
                                         row_bytes, size_t(n), hipMemcpyHostToDevice);
    auto t1 = clock::now();
    if (e != hipSuccess) rs = set_hip_error(e, "record copy");
    if (rs == DT_OK) {
        e = hipEventRecord(s.ev[kEvKernel], s.stream);
        if (e == hipSuccess) rs = classify(d_x, n, d_out, s.stream);
        if (e == hipSuccess && rs == DT_OK) e = hipEventRecord(s.ev[kEvOut], s.stream);
        if (e == hipSuccess && rs == DT_OK) e = hipStreamSynchronize(s.stream);
        if (e != hipSuccess && rs == DT_OK) rs = set_hip_error(e, "classify");
        if (rs == DT_OK) st->kernel_us = elapsed_us(s.ev[kEvKernel], s.ev[kEvOut]);
    }
    auto t2 = clock::now();
    if (rs == DT_OK) {
        e = hipMemcpy(h_out, d_out, size_t(n * esize), hipMemcpyDeviceToHost);
        if (e != hipSuccess) rs = set_hip_error(e, "label copy");
    }
    auto t3 = clock::now();
    (void)hipStreamSynchronize(s.stream);
    (void)hipFree(d_x);
    (void)hipFree(d_out);
    st->h2d_us = std::chrono::duration<double, std::micro>(t1 - t0).count();
    st->d2h_us = std::chrono::duration<double, std::micro>(t3 - t2).count();
    return rs;
}

template <class Obj>
dt_status classify_host(const Obj *obj, dt_pipeline *p, const void *h_x, dt_dtype x_type,
                        int64_t n, int64_t ld, void *h_out, dt_output out_kind,
                        const ClassifyFn &classify, dt_pipeline_stats *stats) {
    using clock = std::chrono::steady_clock;
    const auto t0 = clock::now();
    dt_pipeline_stats st{};
    if (!obj) return set_error(DT_ERR_INVALID_ARG, "tree or forest is NULL");
    if (!p) return set_error(DT_ERR_INVALID_ARG, "pipeline is NULL");
    if (dtree::features_of(obj) != p->n_features)
        return set_error(DT_ERR_INVALID_ARG, "the pipeline was created for another n_features");
    if (dtree::device_of(obj) != p->device)
        return set_error(DT_ERR_INVALID_ARG, "the pipeline and the tree are on different devices");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return set_hip_error(e, "hipGetDevice");
    if (dev != p->device)
        return set_error(DT_ERR_INVALID_ARG, "current device differs from the pipeline's device");
    if (n < 0) return set_error(DT_ERR_INVALID_ARG, "n must be >= 0");
    if (ld < p->n_features) return set_error(DT_ERR_INVALID_ARG, "ld must be >= n_features");
    if (n > kMaxRows) return set_error(DT_ERR_UNSUPPORTED, "n > 2^37");
    // argument checks of the classify call itself (algo, out_kind, classes) on no records
    dt_status rs = classify(nullptr, 0, nullptr, p->slots[0].stream);
    if (rs != DT_OK) return rs;
    if (n > 0 && (!h_x || !h_out)) return set_error(DT_ERR_INVALID_ARG, "null host pointer");
    const int xsize = x_type == DT_F32 ? 4 : x_type == DT_U8 ? 1 : 2;
    if ((reinterpret_cast<uintptr_t>(h_x) % uintptr_t(xsize)) != 0)
        return set_error(DT_ERR_INVALID_ARG, "h_x is not aligned to its element size");
    const int esize = out_kind == DT_OUT_CLASS_U8 ? 1 : 4;
    auto *out = static_cast<unsigned char *>(h_out);
    const char *x = static_cast<const char *>(h_x);
    if (n > 0)
        rs = p->serial ? run_serial(p, classify, x, xsize, n, ld, out, esize, &st)
                       : run_chunked(p, classify, x, xsize, n, ld, out, esize, &st);
    st.outer_us = std::chrono::duration<double, std::micro>(clock::now() - t0).count();
    if (stats) *stats = st;
    return rs;
}

// ---- no-allocation variant of dt_classify_host -------------------------------------------
// For callers that cannot allocate: the records are staged through `scratch`, a fixed
// array of the library's code object (one copy per device, held until the process ends),
// in chunks, one after the other on the caller's stream.
constexpr int64_t kNoAllocScratchBytes = DT_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

// Device address of `scratch` on each device, looked up once per device (with that device
// current) and kept: in host code `scratch` names a host-side stand-in, not device memory.
constexpr int kMaxDevices = 64;
std::atomic<unsigned char *> g_scratch[kMaxDevices];
std::mutex g_scratch_mutex;

dt_status scratch_on(int dev, unsigned char **out) {
    if (dev < 0 || dev >= kMaxDevices) return set_error(DT_ERR_UNSUPPORTED, "device index >= 64");
    unsigned char *p = g_scratch[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mutex);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (!p) {
            void *addr = nullptr;
            const hipError_t e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return set_hip_error(e, "hipGetSymbolAddress(scratch)");
            p = static_cast<unsigned char *>(addr);
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return DT_OK;
}

dt_status classify_host_noalloc(const dt_tree *tree, const float *h_x, int64_t n, int64_t ld,
                                void *h_out, dt_output out_kind, dt_algo algo,
                                hipStream_t stream) {
    if (!tree) return set_error(DT_ERR_INVALID_ARG, "tree is NULL");
    const int32_t F = dtree::features_of(tree);
    if (n < 0) return set_error(DT_ERR_INVALID_ARG, "n must be >= 0");
    if (ld < F) return set_error(DT_ERR_INVALID_ARG, "ld must be >= n_features");
    if (n > kMaxRows) return set_error(DT_ERR_UNSUPPORTED, "n > 2^37");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return set_hip_error(e, "hipGetDevice");
    if (dev != dtree::device_of(tree))
        return set_error(DT_ERR_INVALID_ARG, "current device differs from the tree's device");
    unsigned char *base = nullptr;
    dt_status rs = scratch_on(dev, &base);
    if (rs != DT_OK) return rs;
    // argument checks of the classify call itself (algo, out_kind, classes) on no records
    rs = dt_classify(tree, reinterpret_cast<const float *>(base), 0, F, base, out_kind, algo,
                     stream);
    if (rs != DT_OK || n == 0) return rs;
    if (!h_x || !h_out) return set_error(DT_ERR_INVALID_ARG, "null host pointer");
    if (F > kMaxFeatures) return set_error(DT_ERR_UNSUPPORTED, "n_features > 256");
    // chunk layout in the staging area: dense records (chunk_rows x F floats), then labels
    const int esize = out_kind == DT_OUT_CLASS_U8 ? 1 : 4;
    const int64_t row_bytes = int64_t(F) * 4;
    const int64_t chunk_rows = (kNoAllocScratchBytes - 256) / (row_bytes + esize) / 64 * 64;
    const int64_t label_off = (chunk_rows * row_bytes + 255) / 256 * 256;
    float *d_x = reinterpret_cast<float *>(base);
    unsigned char *d_out = base + label_off;
    const char *hx = reinterpret_cast<const char *>(h_x);
    unsigned char *ho = static_cast<unsigned char *>(h_out);
    for (int64_t r0 = 0; r0 < n; r0 += chunk_rows) {
        const int64_t rows = std::min(chunk_rows, n - r0);
        e = hipMemcpy2DAsync(d_x, size_t(row_bytes), hx + r0 * ld * 4, size_t(ld * 4),
                             size_t(row_bytes), size_t(rows), hipMemcpyHostToDevice, stream);
        if (e != hipSuccess) rs = set_hip_error(e, "hipMemcpy2DAsync(records)");
        if (rs == DT_OK) rs = dt_classify(tree, d_x, rows, F, d_out, out_kind, algo, stream);
        if (rs == DT_OK) {
            e = hipMemcpyAsync(ho + r0 * esize, d_out, size_t(rows * esize),
                               hipMemcpyDeviceToHost, stream);
            if (e != hipSuccess) rs = set_hip_error(e, "hipMemcpyAsync(labels)");
        }
        if (rs != DT_OK) break;
    }
    // synchronous: the labels are in h_out, and no copy or kernel of the call is left
    // running, on success or error
    e = hipStreamSynchronize(stream);
    if (rs == DT_OK && e != hipSuccess) rs = set_hip_error(e, "hipStreamSynchronize");
    return rs;
}

}  // namespace

extern "C" {

dt_status dt_classify_host_noalloc(const dt_tree *tree, const float *h_x, int64_t n, int64_t ld,
                                   void *h_out, dt_output out_kind, dt_algo algo, void *stream) {
    try {
        dtree::clear_error();
        return classify_host_noalloc(tree, h_x, n, ld, h_out, out_kind, algo,
                                     static_cast<hipStream_t>(stream));
    } catch (...) {
        return set_error(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

int64_t dt_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

dt_status dt_pipeline_create(int32_t n_features, const dt_pipeline_options *opt,
                             dt_pipeline **out) {
    try {
        dtree::clear_error();
        return create_impl(n_features, opt, out);
    } catch (const std::bad_alloc &) {
        return set_error(DT_ERR_NO_MEMORY, "host allocation failed");
    } catch (...) {
        return set_error(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

void dt_pipeline_destroy(dt_pipeline *pipeline) {
    if (!pipeline) return;
    release(pipeline);
    delete pipeline;
}

dt_status dt_classify_host(const dt_tree *tree, dt_pipeline *pipeline, const float *h_x,
                           int64_t n, int64_t ld, void *h_out, dt_output out_kind,
                           dt_algo algo, dt_pipeline_stats *stats) {
    try {
        dtree::clear_error();
        const int32_t F = pipeline ? pipeline->n_features : 0;
        const ClassifyFn fn = [=](const void *d_x, int64_t rows, void *d_out, hipStream_t s) {
            return dt_classify(tree, static_cast<const float *>(d_x), rows, F, d_out, out_kind,
                               algo, s);
        };
        return classify_host(tree, pipeline, h_x, DT_F32, n, ld, h_out, out_kind, fn, stats);
    } catch (...) {
        if (pipeline) drain(pipeline);
        return set_error(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

dt_status dt_forest_classify_host(const dt_forest *forest, dt_pipeline *pipeline,
                                  const float *h_x, int64_t n, int64_t ld, void *h_out,
                                  dt_output out_kind, dt_algo algo, dt_pipeline_stats *stats) {
    try {
        dtree::clear_error();
        const int32_t F = pipeline ? pipeline->n_features : 0;
        const ClassifyFn fn = [=](const void *d_x, int64_t rows, void *d_out, hipStream_t s) {
            return dt_forest_classify(forest, static_cast<const float *>(d_x), rows, F, d_out,
                                      out_kind, algo, s);
        };
        return classify_host(forest, pipeline, h_x, DT_F32, n, ld, h_out, out_kind, fn, stats);
    } catch (...) {
        if (pipeline) drain(pipeline);
        return set_error(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

dt_status dt_classify_host_typed(const dt_tree *tree, dt_pipeline *pipeline, const void *h_x,
                                 dt_dtype x_type, int64_t n, int64_t ld, void *h_out,
                                 dt_output out_kind, dt_algo algo, dt_pipeline_stats *stats) {
    try {
        dtree::clear_error();
        if (x_type != DT_F32 && x_type != DT_F16 && x_type != DT_BF16 && x_type != DT_U8)
            return set_error(DT_ERR_INVALID_ARG, "unknown x_type");
        const int32_t F = pipeline ? pipeline->n_features : 0;
        const ClassifyFn fn = [=](const void *d_x, int64_t rows, void *d_out, hipStream_t s) {
            return dt_classify_typed(tree, d_x, x_type, rows, F, d_out, out_kind, algo, s);
        };
        return classify_host(tree, pipeline, h_x, x_type, n, ld, h_out, out_kind, fn, stats);
    } catch (...) {
        if (pipeline) drain(pipeline);
        return set_error(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

}  // extern "C"
