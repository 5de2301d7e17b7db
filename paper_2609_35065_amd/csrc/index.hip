// index.hip -- the staged-chunk index: key -> staging slot.
//
// Host policy decides what is staged (job build allocates slots, eviction
// frees them), so the authoritative table lives on the host (IndexTable,
// index_table.cpp); kv_lookup probes a device mirror of it.  Both use the same
// open-addressing layout, so a mutation is mirrored by uploading the table
// image.
//
// Uploads are stream-ordered, so a lookup enqueued after an insert on the
// same stream sees the insert.  A mutation that changed few entries uploads
// only those: (position, entry) pairs go through a pinned snapshot buffer to
// a device list, and a small kernel writes them into the table.  After a
// rehash, or when many entries changed, the whole table image is sent
// instead.  Each of the two snapshot buffers (and its device list) is reused
// only after the event recorded behind its previous upload has completed.

#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <vector>

#include "internal.h"

namespace tkv {
// One changed table entry, as uploaded by an incremental update.
struct alignas(16) IndexUpdate {
    int64_t pos;
    int64_t pad;
    IndexEntry entry;
};
}  // namespace tkv

struct kv_index {
    int device = 0;
    tkv::IndexTable table;           // the authoritative host table
    tkv::IndexEntry *dev = nullptr;  // its device mirror
    tkv::IndexEntry *snap[2] = {nullptr, nullptr};
    tkv::IndexUpdate *dev_upd[2] = {nullptr, nullptr};
    int64_t upd_cap = 0;             // pairs per incremental upload
    hipEvent_t ev[2] = {nullptr, nullptr};
    bool ev_used[2] = {false, false};
    int next = 0;
};

namespace {

using tkv::IndexEntry;
using tkv::IndexUpdate;

constexpr int kApplyThreads = 256;

__global__ __launch_bounds__(kApplyThreads) void index_apply_kernel(const IndexUpdate *__restrict__ upd, int64_t n,
                                                                   int64_t cap, IndexEntry *__restrict__ table) {
    const int64_t i = (int64_t)blockIdx.x * kApplyThreads + threadIdx.x;
    if (i >= n) return;
    const int64_t pos = upd[i].pos;
    if (pos >= 0 && pos < cap) table[pos] = upd[i].entry;
}

// Mirror the host mutations since the last upload into the device table.  An
// incremental update stages its (position, entry) pairs in `upd_list`, a
// device buffer of `upd_pairs` pairs; more changes than that, or a rebuilt
// table, send the whole table image.
int upload_via(kv_index *ix, hipStream_t stream, IndexUpdate *upd_list, int64_t upd_pairs) {
    tkv::IndexTable &t = ix->table;
    int prev = 0;
    if (hipGetDevice(&prev) != hipSuccess) return KV_EHIP;
    if (prev != ix->device && hipSetDevice(ix->device) != hipSuccess) return KV_EHIP;
    int rc = KV_OK;
    const int k = ix->next;
    const size_t bytes = sizeof(IndexEntry) * (size_t)t.cap;
    if (ix->ev_used[k] && hipEventSynchronize(ix->ev[k]) != hipSuccess) rc = KV_EHIP;
    const std::vector<int64_t> &dirty = t.changes();
    const int64_t n = (int64_t)dirty.size();
    if (rc == KV_OK && (t.rebuilt || n > upd_pairs)) {
        memcpy(ix->snap[k], t.entries.data(), bytes);
        if (hipMemcpyAsync(ix->dev, ix->snap[k], bytes, hipMemcpyHostToDevice, stream) != hipSuccess ||
            hipEventRecord(ix->ev[k], stream) != hipSuccess)
            rc = KV_EHIP;
        else
            ix->ev_used[k] = true;
    } else if (rc == KV_OK && n > 0) {
        IndexUpdate *list = reinterpret_cast<IndexUpdate *>(ix->snap[k]);
        for (int64_t i = 0; i < n; ++i) list[i] = IndexUpdate{dirty[i], 0, t.entries[dirty[i]]};
        (void)hipGetLastError();
        if (hipMemcpyAsync(upd_list, list, sizeof(IndexUpdate) * (size_t)n, hipMemcpyHostToDevice, stream) !=
            hipSuccess) {
            rc = KV_EHIP;
        } else {
            hipLaunchKernelGGL(index_apply_kernel, dim3((unsigned)((n + kApplyThreads - 1) / kApplyThreads)),
                               dim3(kApplyThreads), 0, stream, upd_list, n, t.cap, ix->dev);
            if (hipGetLastError() != hipSuccess || hipEventRecord(ix->ev[k], stream) != hipSuccess)
                rc = KV_EHIP;
            else
                ix->ev_used[k] = true;
        }
    }
    if (rc == KV_OK) {
        t.rebuilt = false;
        t.clear_changes();
    }
    ix->next = k ^ 1;
    if (prev != ix->device) (void)hipSetDevice(prev);
    return rc;
}

int upload(kv_index *ix, hipStream_t stream) { return upload_via(ix, stream, ix->dev_upd[ix->next], ix->upd_cap); }

// --------------------------------------------------------------------------
// Allocation-free insert (kv_index_insert_static): the pairs of an
// incremental update are staged in `scratch`, a fixed device array, instead
// of the index's own device lists.  Each GPU holds its own copy of the array;
// its address on a device is taken once, with that device current, and only
// that address is handed to copies and kernels.  Every call on one GPU uses
// the same array, so such calls must be ordered on one stream.
// --------------------------------------------------------------------------
constexpr int64_t kStaticPairs = KV_INDEX_STATIC_MAX_PAIRS;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) IndexUpdate scratch[kStaticPairs];

std::mutex g_scratch_mu;
IndexUpdate *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on `device`, which must be the current device,
// or nullptr.  Taken once per device (by kv_index_create, the first call that
// can need it there) and cached.
IndexUpdate *scratch_on(int device) {
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
            (void)hipGetLastError();
            return nullptr;
        }
        g_scratch_ptr[device] = static_cast<IndexUpdate *>(ptr);
    }
    return g_scratch_ptr[device];
}

void release(kv_index *ix) {
    for (int k = 0; k < 2; ++k) {
        if (ix->ev[k]) {
            (void)hipEventSynchronize(ix->ev[k]);
            (void)hipEventDestroy(ix->ev[k]);
        }
        if (ix->snap[k]) (void)hipHostFree(ix->snap[k]);
        if (ix->dev_upd[k]) (void)hipFree(ix->dev_upd[k]);
    }
    if (ix->dev) (void)hipFree(ix->dev);
    delete ix;
}

}  // namespace

namespace tkv {
const IndexEntry *index_device_table(const kv_index *idx, int *log2cap) {
    *log2cap = idx->table.log2cap;
    return idx->dev;
}
}  // namespace tkv

extern "C" {

int kv_index_create(int64_t max_entries, kv_index **out) {
    if (!out || max_entries <= 0 || max_entries > (int64_t(1) << 28)) return KV_EINVAL;
    *out = nullptr;
    kv_index *ix = new (std::nothrow) kv_index();
    if (!ix) return KV_EINVAL;
    // changed positions between uploads: room for the largest allocation-free insert, and then some
    if (!ix->table.init(max_entries, 2 * KV_INDEX_STATIC_MAX_PAIRS)) {
        delete ix;
        return KV_EINVAL;
    }
    const int64_t cap = ix->table.cap;
    const size_t bytes = sizeof(IndexEntry) * (size_t)cap;
    // an incremental upload fits a snapshot buffer (cap entries = cap/2 pairs); past an eighth of the
    // table, or 65536 pairs, the whole image is sent instead
    ix->upd_cap = std::min<int64_t>(cap / 8, 65536);
    const size_t upd_bytes = sizeof(IndexUpdate) * (size_t)ix->upd_cap;
    if (hipGetDevice(&ix->device) != hipSuccess || hipMalloc((void **)&ix->dev, bytes) != hipSuccess ||
        hipMalloc((void **)&ix->dev_upd[0], upd_bytes) != hipSuccess ||
        hipMalloc((void **)&ix->dev_upd[1], upd_bytes) != hipSuccess ||
        hipMemset(ix->dev, 0, bytes) != hipSuccess ||
        hipHostMalloc((void **)&ix->snap[0], bytes, hipHostMallocDefault) != hipSuccess ||
        hipHostMalloc((void **)&ix->snap[1], bytes, hipHostMallocDefault) != hipSuccess ||
        hipEventCreateWithFlags(&ix->ev[0], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&ix->ev[1], hipEventDisableTiming) != hipSuccess ||
        !scratch_on(ix->device) ||   // set-up of kv_index_insert_static on this device
        hipDeviceSynchronize() != hipSuccess) {
        release(ix);
        return KV_EHIP;
    }
    *out = ix;
    return KV_OK;
}

int kv_index_destroy(kv_index *idx) {
    if (!idx) return KV_EINVAL;
    release(idx);
    return KV_OK;
}

int kv_index_insert(kv_index *idx, const uint64_t *h_keys, const int32_t *h_slots, int32_t n, void *stream) {
    if (!idx || n < 0 || (n > 0 && (!h_keys || !h_slots))) return KV_EINVAL;
    for (int32_t i = 0; i < n; ++i)
        if (h_slots[i] < 0) return KV_EINVAL;
    const int rc = idx->table.insert(h_keys, h_slots, n);
    const int up = upload(idx, (hipStream_t)stream);
    return rc != KV_OK ? rc : up;
}

int kv_index_insert_static(kv_index *idx, const uint64_t *h_keys, const int32_t *h_slots, int32_t n,
                           void *stream) {
    if (!idx || n < 0 || (n > 0 && (!h_keys || !h_slots))) return KV_EINVAL;
    if (n > kStaticPairs) return KV_ELIMIT;
    for (int32_t i = 0; i < n; ++i)
        if (h_slots[i] < 0) return KV_EINVAL;
    int prev = 0;
    if (hipGetDevice(&prev) != hipSuccess) return KV_EHIP;
    if (prev != idx->device && hipSetDevice(idx->device) != hipSuccess) return KV_EHIP;
    IndexUpdate *list = scratch_on(idx->device);
    if (prev != idx->device) (void)hipSetDevice(prev);
    if (!list) return KV_EHIP;
    const int rc = idx->table.insert(h_keys, h_slots, n);
    const int up = upload_via(idx, (hipStream_t)stream, list, std::min<int64_t>(idx->upd_cap, kStaticPairs));
    return rc != KV_OK ? rc : up;
}

int kv_index_erase(kv_index *idx, const uint64_t *h_keys, int32_t n, void *stream) {
    if (!idx || n < 0 || (n > 0 && !h_keys)) return KV_EINVAL;
    idx->table.erase(h_keys, n);
    return upload(idx, (hipStream_t)stream);
}

int kv_index_size(const kv_index *idx, int64_t *out) {
    if (!idx || !out) return KV_EINVAL;
    *out = idx->table.live;
    return KV_OK;
}

int kv_index_find(const kv_index *idx, uint64_t key, int32_t *slot_out) {
    if (!idx || !slot_out) return KV_EINVAL;
    *slot_out = idx->table.find(key);
    return KV_OK;
}

}  // extern "C"
