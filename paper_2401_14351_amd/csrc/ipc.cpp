// Handoff of a loaded device buffer to another process (Sec. 4.1: the
// inference process gets the GPU base address from the model manager as an
// IPC handle, adds the tensor offsets from the index, and synchronizes with
// the manager).  The synchronization is an interprocess event recorded after
// the load: the importer's stream waits for it on the device.
#include <cstring>

#include "hip_util.hpp"

using namespace sllm;

static_assert(sizeof(hipIpcMemHandle_t) == 64, "IPC memory handle size");
static_assert(sizeof(hipIpcEventHandle_t) == 64, "IPC event handle size");

struct sllm_export {
    int device = 0;
    hipEvent_t ev = nullptr;
};

struct sllm_import {
    int device = 0;
    void* base = nullptr;
    hipEvent_t ev = nullptr;
};

extern "C" int32_t sllm_export_create(const void* dev_ptr, uint64_t bytes, int32_t device, void* stream,
                                      sllm_ipc_desc* desc, sllm_export** out) try {
    clear_error();
    if (!dev_ptr || !desc || !out) return fail(SLLM_E_INVAL, "dev_ptr, desc and out must be non-NULL");
    *out = nullptr;
    DeviceGuard guard(device);
    if (!guard.ok()) return fail(SLLM_E_HIP, "cannot make device %d current", device);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void*>(dev_ptr)) != hipSuccess || !base)
        return fail(SLLM_E_INVAL, "%p is not device memory", dev_ptr);
    const uint64_t off = (uint64_t)((const uint8_t*)dev_ptr - (const uint8_t*)base);
    if (bytes > size || off > size - bytes) return fail(SLLM_E_INVAL, "range runs past its allocation");
    if (size > SLLM_IPC_MAX_ALLOCATION)
        return fail(SLLM_E_INVAL, "allocation of %zu bytes is larger than the %llu bytes shared across processes", size,
                    (unsigned long long)SLLM_IPC_MAX_ALLOCATION);
    hipIpcMemHandle_t mh;
    SLLM_HIP(hipIpcGetMemHandle(&mh, base));
    auto* ex = new (std::nothrow) sllm_export;
    if (!ex) return fail(SLLM_E_NOMEM, "out of host memory");
    ex->device = device;
    std::memset(desc, 0, sizeof *desc);
    hipStream_t s = static_cast<hipStream_t>(stream);
    // preferred: an interprocess event the importer's stream waits on
    hipIpcEventHandle_t eh;
    const char* what = "hipEventCreateWithFlags(interprocess)";
    hipError_t e = hipEventCreateWithFlags(&ex->ev, hipEventDisableTiming | hipEventInterprocess);
    if (e == hipSuccess) {
        what = "hipIpcGetEventHandle";
        e = hipIpcGetEventHandle(&eh, ex->ev);
    }
    if (e == hipSuccess) {
        what = "hipEventRecord";
        e = hipEventRecord(ex->ev, s);
        if (e != hipSuccess) {
            (void)hipEventDestroy(ex->ev);
            delete ex;
            return fail(SLLM_E_HIP, "%s: %s", what, hipGetErrorString(e));
        }
        std::memcpy(desc->event_handle, &eh, sizeof eh);
        desc->flags |= SLLM_IPC_HAS_EVENT;
    } else {
        // no interprocess events here: finish the load before handing out the buffer
        log_msg(1, "%s failed (%s); the export synchronizes on the host instead", what, hipGetErrorString(e));
        if (ex->ev) (void)hipEventDestroy(ex->ev);
        ex->ev = nullptr;
        (void)hipGetLastError();
        e = hipStreamSynchronize(s);
        if (e != hipSuccess) {
            delete ex;
            return fail(SLLM_E_HIP, "hipStreamSynchronize: %s", hipGetErrorString(e));
        }
    }
    std::memcpy(desc->mem_handle, &mh, sizeof mh);
    desc->offset = off;
    desc->bytes = bytes;
    desc->device = device;
    *out = ex;
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_export_destroy(sllm_export* ex) try {
    clear_error();
    if (!ex) return SLLM_OK;
    DeviceGuard guard(ex->device);
    if (ex->ev) (void)hipEventDestroy(ex->ev);
    delete ex;
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_import_open(const sllm_ipc_desc* desc, void* stream, void** dev_ptr, sllm_import** out) try {
    clear_error();
    if (!desc || !dev_ptr || !out) return fail(SLLM_E_INVAL, "desc, dev_ptr and out must be non-NULL");
    *out = nullptr;
    DeviceGuard guard(desc->device);
    if (!guard.ok()) return fail(SLLM_E_HIP, "cannot make device %d current", desc->device);
    auto* im = new (std::nothrow) sllm_import;
    if (!im) return fail(SLLM_E_NOMEM, "out of host memory");
    im->device = desc->device;
    hipIpcMemHandle_t mh;
    hipIpcEventHandle_t eh;
    std::memcpy(&mh, desc->mem_handle, sizeof mh);
    std::memcpy(&eh, desc->event_handle, sizeof eh);
    if (desc->flags & ~SLLM_IPC_HAS_EVENT) {
        delete im;
        return fail(SLLM_E_INVAL, "unknown descriptor flags 0x%x", desc->flags);
    }
    const char* what = "hipIpcOpenMemHandle";
    hipError_t e = hipIpcOpenMemHandle(&im->base, mh, hipIpcMemLazyEnablePeerAccess);
    if (e == hipSuccess && (desc->flags & SLLM_IPC_HAS_EVENT)) {
        what = "hipIpcOpenEventHandle";
        e = hipIpcOpenEventHandle(&im->ev, eh);
        if (e == hipSuccess) {
            what = "hipStreamWaitEvent";
            e = hipStreamWaitEvent(static_cast<hipStream_t>(stream), im->ev, 0);
        }
    }
    int32_t code = SLLM_E_HIP;
    if (e == hipSuccess) {
        // the descriptor comes from another process: its range must lie in
        // the allocation the handle mapped, or views past it would fault
        hipDeviceptr_t base = nullptr;
        size_t size = 0;
        what = "hipMemGetAddressRange";
        e = hipMemGetAddressRange(&base, &size, im->base);
        if (e == hipSuccess && (desc->bytes > size || desc->offset > size - desc->bytes)) {
            code = SLLM_E_INVAL;
            what = "the descriptor's range runs past the shared allocation";
            e = hipErrorInvalidValue;
        }
    }
    if (e != hipSuccess) {
        if (im->ev) (void)hipEventDestroy(im->ev);
        if (im->base) (void)hipIpcCloseMemHandle(im->base);
        delete im;
        return fail(code, "%s: %s", what, hipGetErrorString(e));
    }
    *dev_ptr = static_cast<uint8_t*>(im->base) + desc->offset;
    *out = im;
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_import_close(sllm_import* im) try {
    clear_error();
    if (!im) return SLLM_OK;
    DeviceGuard guard(im->device);
    if (im->ev) (void)hipEventDestroy(im->ev);
    hipError_t e = im->base ? hipIpcCloseMemHandle(im->base) : hipSuccess;
    delete im;
    if (e != hipSuccess) return fail(SLLM_E_HIP, "hipIpcCloseMemHandle: %s", hipGetErrorString(e));
    return SLLM_OK;
} SLLM_CATCH_ALL
