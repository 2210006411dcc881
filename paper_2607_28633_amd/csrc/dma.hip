// Layer shipper: copies each packed layer off the GPU on a DMA (SDMA) engine
// as soon as the stream event that produced it has completed, so the transfer
// of layer l proceeds while layers l+1 .. L of the prefill keep every compute
// unit (Sec. 5.2: layer l is sent while later layers still compute).
//
// HIP's own device-to-host copy into pinned memory runs as a copy kernel on
// the compute units; behind a prefill kernel that occupies all of them it only
// gets a unit when one of the prefill's workgroups retires.  ROCr's
// hsa_amd_memory_async_copy drives the GPU's DMA engines instead and uses no
// compute unit.  A host worker thread turns "event completed" into "start the
// copy" (HIP events are not HSA signals), keeping up to kInFlight copies
// outstanding; tickets complete in submission order.  The receiving side
// uses the same path the other way round: pinned host memory into device
// memory, each layer unpacked once its ticket has completed.
#include <hip/hip_runtime.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <condition_variable>
#include <cstdint>
#include <deque>
#include <mutex>
#include <new>
#include <thread>

#include "topkv.h"

namespace {

constexpr int kInFlight = 2;

struct Item {
    hipEvent_t ready;
    void* dst;
    const void* src;
    size_t bytes;
    hsa_agent_t dst_agent, src_agent;
    int64_t ticket;
};

struct Flight {
    hsa_signal_t signal;
    int64_t ticket;
};

// The allocation that holds [p, p + bytes), and the agent that owns it.
bool locate(const void* p, size_t bytes, hsa_agent_t* owner) {
    hsa_amd_pointer_info_t info = {};
    info.size = sizeof(info);
    if (hsa_amd_pointer_info(p, &info, nullptr, nullptr, nullptr) != HSA_STATUS_SUCCESS) return false;
    if (info.type != HSA_EXT_POINTER_TYPE_HSA) return false;    // hipMalloc / hipHostMalloc memory
    const uintptr_t base = reinterpret_cast<uintptr_t>(info.agentBaseAddress);
    const uintptr_t at = reinterpret_cast<uintptr_t>(p);
    if (at < base || at - base > info.sizeInBytes || bytes > info.sizeInBytes - (at - base)) return false;
    *owner = info.agentOwner;
    return true;
}

}  // namespace

struct topkv_dma {
    std::mutex mu;
    std::condition_variable work, done;
    std::deque<Item> queue;
    int64_t next_ticket = 1, completed = 0;
    topkv_status_t status = TOPKV_OK;
    bool stop = false;
    int device = 0;
    hsa_signal_t signals[kInFlight] = {};
    std::thread worker;

    void fail(topkv_status_t st) {
        if (status == TOPKV_OK) status = st;
        queue.clear();
        done.notify_all();
    }

    // Wait for the oldest outstanding copy (called and returning with mu held).
    void retire(std::unique_lock<std::mutex>& lk, std::deque<Flight>& flight) {
        const Flight f = flight.front();
        flight.pop_front();
        lk.unlock();
        const hsa_signal_value_t v = hsa_signal_wait_scacquire(f.signal, HSA_SIGNAL_CONDITION_LT, 1,
                                                               UINT64_MAX, HSA_WAIT_STATE_BLOCKED);
        lk.lock();
        if (v != 0) fail(TOPKV_ERR_DEVICE);
        else if (status == TOPKV_OK) completed = f.ticket;
        done.notify_all();
    }

    void run() {
        (void)hipSetDevice(device);          // events of another device still synchronise
        std::deque<Flight> flight;
        int slot = 0;                 // signals are used round robin, retired in FIFO order
        std::unique_lock<std::mutex> lk(mu);
        for (;;) {
            if (queue.empty()) {
                if (!flight.empty()) { retire(lk, flight); continue; }
                if (stop) break;
                work.wait(lk, [&] { return stop || !queue.empty(); });
                continue;
            }
            const Item it = queue.front();
            queue.pop_front();
            if (it.bytes == 0) {          // nothing to copy: completes after everything before it
                while (!flight.empty()) retire(lk, flight);
            } else if (static_cast<int>(flight.size()) == kInFlight) {
                retire(lk, flight);
            }
            if (status != TOPKV_OK) continue;
            lk.unlock();
            bool ok = !it.ready || hipEventSynchronize(it.ready) == hipSuccess;
            const hsa_signal_t sig = signals[slot];
            if (ok && it.bytes) {
                hsa_signal_store_screlease(sig, 1);
                ok = hsa_amd_memory_async_copy(it.dst, it.dst_agent, it.src, it.src_agent, it.bytes, 0,
                                               nullptr, sig) == HSA_STATUS_SUCCESS;
            }
            lk.lock();
            if (!ok) {
                fail(TOPKV_ERR_DEVICE);
            } else if (it.bytes == 0) {
                completed = it.ticket;
                done.notify_all();
            } else {
                flight.push_back({sig, it.ticket});
                slot = (slot + 1) % kInFlight;
            }
        }
    }
};

extern "C" {

topkv_status_t topkv_dma_create(topkv_dma_t** out) {
    if (!out) return TOPKV_ERR_INVALID_ARG;
    *out = nullptr;
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return TOPKV_ERR_DEVICE;
    if (hsa_init() != HSA_STATUS_SUCCESS) return TOPKV_ERR_DEVICE;
    topkv_dma* d = new (std::nothrow) topkv_dma();
    if (!d) { hsa_shut_down(); return TOPKV_ERR_DEVICE; }
    d->device = device;
    for (int i = 0; i < kInFlight; ++i) {
        if (hsa_signal_create(0, 0, nullptr, &d->signals[i]) != HSA_STATUS_SUCCESS) {
            for (int j = 0; j < i; ++j) hsa_signal_destroy(d->signals[j]);
            delete d;
            hsa_shut_down();
            return TOPKV_ERR_DEVICE;
        }
    }
    d->worker = std::thread([d] { d->run(); });
    *out = d;
    return TOPKV_OK;
}

topkv_status_t topkv_dma_submit(topkv_dma_t* dma, hipEvent_t ready, void* dst, const void* src,
                                int64_t bytes, int64_t* ticket) {
    if (!dma || !ticket || bytes < 0 || (bytes > 0 && (!dst || !src))) return TOPKV_ERR_INVALID_ARG;
    Item it = {ready, dst, src, static_cast<size_t>(bytes), {}, {}, 0};
    if (bytes > 0 && (!locate(dst, it.bytes, &it.dst_agent) || !locate(src, it.bytes, &it.src_agent)))
        return TOPKV_ERR_BOUNDS;
    std::unique_lock<std::mutex> lk(dma->mu);
    if (dma->status != TOPKV_OK) return dma->status;
    if (dma->stop) return TOPKV_ERR_INVALID_ARG;
    it.ticket = dma->next_ticket++;
    *ticket = it.ticket;
    dma->queue.push_back(it);
    dma->work.notify_one();
    return TOPKV_OK;
}

topkv_status_t topkv_dma_wait(topkv_dma_t* dma, int64_t ticket) {
    if (!dma || ticket < 0) return TOPKV_ERR_INVALID_ARG;
    std::unique_lock<std::mutex> lk(dma->mu);
    if (ticket >= dma->next_ticket) return TOPKV_ERR_INVALID_ARG;
    dma->done.wait(lk, [&] { return dma->completed >= ticket || dma->status != TOPKV_OK; });
    return dma->completed >= ticket ? TOPKV_OK : dma->status;
}

topkv_status_t topkv_dma_destroy(topkv_dma_t* dma) {
    if (!dma) return TOPKV_ERR_INVALID_ARG;
    {
        std::lock_guard<std::mutex> lk(dma->mu);
        dma->stop = true;
    }
    dma->work.notify_all();
    dma->worker.join();
    const topkv_status_t st = dma->status;
    for (int i = 0; i < kInFlight; ++i) hsa_signal_destroy(dma->signals[i]);
    delete dma;
    hsa_shut_down();
    return st;
}

}  // extern "C"
