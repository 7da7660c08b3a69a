// Runtime IPC-handle exchange (Zero-SM Point-to-Point Executor, intra-node
// communication): a process exports the allocation that holds one of its
// buffers as an IPC handle plus the buffer's offset in it; another process
// on the same device opens the handle and addresses the buffer directly, so
// a copy engine or a kernel of that process can read or write it.  The
// handles travel between processes out of band (the PyTorch backend posts
// them in a shared-memory mailbox).  Opened handles are cached per handle, so a
// buffer reused call after call is opened once.
#include <hip/hip_runtime.h>

#include <cstring>
#include <map>
#include <mutex>
#include <string>

#include "../../include/hoccl.h"

namespace hoccl {
namespace {

// Opening an exported allocation of 2 GiB or more has not returned on these
// machines; such allocations are refused rather than risked.
constexpr size_t kMaxIpcBytes = (size_t)2 << 30;

struct Opened {
    void *base;
    size_t bytes;
};

std::mutex g_ipc_mu;
std::map<std::string, Opened> g_opened;  // handle bytes -> mapping

}  // namespace
}  // namespace hoccl

using namespace hoccl;

extern "C" {

hoccl_status_t hoccl_ipc_export(const void *ptr, void *handle, size_t *offset, size_t *alloc_bytes) {
    if (!ptr || !handle || !offset || !alloc_bytes) return HOCCL_ERR_INVALID_ARG;
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)ptr) != hipSuccess || !base) {
        (void)hipGetLastError();
        return HOCCL_ERR_INVALID_ARG;  // not device memory from an allocation
    }
    if (size >= kMaxIpcBytes) return HOCCL_ERR_UNSUPPORTED;
    hipIpcMemHandle_t h;
    if (hipIpcGetMemHandle(&h, (void *)base) != hipSuccess) {
        (void)hipGetLastError();
        return HOCCL_ERR_HIP;
    }
    std::memcpy(handle, &h, sizeof h);
    *offset = (size_t)((const char *)ptr - (const char *)base);
    *alloc_bytes = size;
    return HOCCL_OK;
}

hoccl_status_t hoccl_ipc_open(const void *handle, size_t offset, size_t alloc_bytes, void **ptr) {
    if (!handle || !ptr || offset >= alloc_bytes) return HOCCL_ERR_INVALID_ARG;
    if (alloc_bytes >= kMaxIpcBytes) return HOCCL_ERR_UNSUPPORTED;
    const std::string key((const char *)handle, HIP_IPC_HANDLE_SIZE);
    std::lock_guard<std::mutex> lk(g_ipc_mu);
    auto it = g_opened.find(key);
    if (it == g_opened.end()) {
        hipIpcMemHandle_t h;
        std::memcpy(&h, handle, sizeof h);
        void *base = nullptr;
        if (hipIpcOpenMemHandle(&base, h, hipIpcMemLazyEnablePeerAccess) != hipSuccess || !base) {
            (void)hipGetLastError();
            return HOCCL_ERR_HIP;
        }
        it = g_opened.emplace(key, Opened{base, alloc_bytes}).first;
    }
    if (offset >= it->second.bytes) return HOCCL_ERR_INVALID_ARG;
    *ptr = (char *)it->second.base + offset;
    return HOCCL_OK;
}

hoccl_status_t hoccl_ipc_close_all(void) {
    std::lock_guard<std::mutex> lk(g_ipc_mu);
    hoccl_status_t st = HOCCL_OK;
    for (auto &kv : g_opened)
        if (hipIpcCloseMemHandle(kv.second.base) != hipSuccess) {
            (void)hipGetLastError();
            st = HOCCL_ERR_HIP;
        }
    g_opened.clear();
    return st;
}

}  // extern "C"
