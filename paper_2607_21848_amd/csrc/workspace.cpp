// Device workspace owned by the library: one block per (device, stream),
// allocated on first use and grown when a call needs more. Calls queued on
// one stream run in order and may share the block; calls on different streams
// get different blocks. Blocks live until the process ends.

#include <stddef.h>

#include <mutex>
#include <new>
#include <vector>

#include <hip/hip_runtime.h>

#include "internal.h"

namespace revisit {

namespace {

struct Block {
    int device;
    hipStream_t stream;
    void* ptr;
    size_t bytes;
};

std::mutex g_mutex;
std::vector<Block> g_blocks;
std::vector<int> g_cus;  // compute units by device, -1 = not queried yet

}  // namespace

hipError_t stream_workspace(hipStream_t stream, size_t bytes, void** out) {
    *out = nullptr;
    if (bytes == 0) return hipSuccess;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(g_mutex);
    for (Block& b : g_blocks) {
        if (b.device != dev || b.stream != stream) continue;
        if (b.bytes < bytes) {
            // work queued earlier on this stream may still use the old block
            e = hipStreamSynchronize(stream);
            if (e != hipSuccess) return e;
            e = hipFree(b.ptr);
            b.ptr = nullptr;
            b.bytes = 0;
            if (e != hipSuccess) return e;
            e = hipMalloc(&b.ptr, bytes);
            if (e != hipSuccess) return e;
            b.bytes = bytes;
        }
        *out = b.ptr;
        return hipSuccess;
    }
    void* p = nullptr;
    e = hipMalloc(&p, bytes);
    if (e != hipSuccess) return e;
    // no C++ exception may leave the library's C entry points
    try {
        g_blocks.push_back(Block{dev, stream, p, bytes});
    } catch (const std::bad_alloc&) {
        (void)hipFree(p);
        return hipErrorOutOfMemory;
    }
    *out = p;
    return hipSuccess;
}

hipError_t device_compute_units(int* cus) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(g_mutex);
    if ((int)g_cus.size() <= dev) {
        try {
            g_cus.resize(dev + 1, -1);
        } catch (const std::bad_alloc&) {
            return hipErrorOutOfMemory;
        }
    }
    if (g_cus[dev] < 0) {
        int n = 0;
        e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        g_cus[dev] = n;
    }
    *cus = g_cus[dev];
    return hipSuccess;
}

}  // namespace revisit
