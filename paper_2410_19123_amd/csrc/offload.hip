// Expert offload for the layer stack (Sec. 4.1): the packed experts of every
// layer live in pinned host memory; a device cache holds (layer, expert)
// slots; a second stream copies the experts of layer l+1 while the compute
// stream runs layer l; misses evict by the Belady rule over the references
// pre-gating makes known (this step's layers, and the next step's when the
// caller passes them), or by LRU.
//
// Ordering.  Per layer l the copy stream records ready[l] after its copies
// and the compute stream waits on it; the compute stream records done[l]
// after the layer's down projection, and before a copy overwrites a slot
// the copy stream waits on done[] of the slot's last layer.  The planner
// (offload_plan.cpp) never overwrites a slot this step used at the layer
// being loaded or at the one before it, whose kernels are enqueued after
// the copy, so a slot is never overwritten while a kernel may still read it.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <vector>

#include "common.hpp"
#include "internal.hpp"
#include "offload_plan.hpp"

using namespace readme;

struct readme_offload {
    int E = 0, L = 0, slots = 0, policy = 0;
    int64_t d = 0, I = 0, Ip = 0;
    size_t gu_bytes = 0, dn_bytes = 0, slot_bytes = 0, layer_bytes = 0;
    std::vector<char*> host;        // pinned, one packed layer each
    char* dev_slots = nullptr;      // slots * slot_bytes: [gate/up | down] per slot
    int32_t* dev_index = nullptr;   // [2][L][E] expert -> slot, by step parity
    int32_t* host_index = nullptr;  // pinned staging of the same
    hipStream_t copy = nullptr;
    std::vector<hipEvent_t> ready, done;
    hipEvent_t table_done[2] = {nullptr, nullptr};
    bool table_used[2] = {false, false};
    OffloadCache cache;              // which (layer, expert) each slot holds
    std::vector<OffloadRef> last_plan;  // the references of the last step
    int64_t hits = 0, misses = 0, bytes = 0;
};

namespace {

void release(readme_offload* ex) {
    if (!ex) return;
    // Nothing may still read or write the slots: the copy stream and the
    // last recorded layer of the compute stream have finished.
    if (ex->copy) (void)hipStreamSynchronize(ex->copy);
    for (hipEvent_t e : ex->done)
        if (e) (void)hipEventSynchronize(e);
    for (char* p : ex->host)
        if (p) (void)hipHostFree(p);
    if (ex->host_index) (void)hipHostFree(ex->host_index);
    if (ex->dev_slots) (void)hipFree(ex->dev_slots);
    if (ex->dev_index) (void)hipFree(ex->dev_index);
    for (hipEvent_t e : ex->ready) (void)hipEventDestroy(e);
    for (hipEvent_t e : ex->done) (void)hipEventDestroy(e);
    for (hipEvent_t e : ex->table_done)
        if (e) (void)hipEventDestroy(e);
    if (ex->copy) (void)hipStreamDestroy(ex->copy);
    delete ex;
}

}  // namespace

extern "C" {

readme_status readme_offload_create(int32_t E, int64_t d, int64_t I, int32_t L, int32_t slots,
                                    int32_t policy, const void* const* packed_layers,
                                    readme_offload** out, void* stream) {
    if (!out) return README_ERR_ARG;
    *out = nullptr;
    if (E < 1 || E > README_MAX_EXPERTS || d <= 0 || d % 64 != 0 || I < 1 || L < 1 || slots < 1)
        return README_ERR_ARG;
    if (policy != README_CACHE_BELADY && policy != README_CACHE_LRU) return README_ERR_ARG;
    if (!packed_layers) return README_ERR_ARG;
    for (int32_t l = 0; l < L; ++l)
        if (!packed_layers[l]) return README_ERR_ARG;
    auto* ex = new readme_offload();
    ex->E = E;
    ex->L = L;
    ex->slots = slots;
    ex->policy = policy;
    ex->d = d;
    ex->I = I;
    ex->Ip = padded_I(I);
    ex->gu_bytes = (size_t)2 * ex->Ip * d * 2;
    ex->dn_bytes = (size_t)d * ex->Ip * 2;
    ex->slot_bytes = ex->gu_bytes + ex->dn_bytes;
    ex->layer_bytes = packed_bytes(README_BF16, E, d, I);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    bool ok = hipStreamCreateWithFlags(&ex->copy, hipStreamNonBlocking) == hipSuccess;
    ex->host.assign(L, nullptr);
    for (int32_t l = 0; ok && l < L; ++l) {
        ok = hipHostMalloc(reinterpret_cast<void**>(&ex->host[l]), ex->layer_bytes,
                           hipHostMallocDefault) == hipSuccess;
        ok = ok && hipMemcpyAsync(ex->host[l], packed_layers[l], ex->layer_bytes,
                                  hipMemcpyDeviceToHost, s) == hipSuccess;
    }
    ok = ok && hipMalloc(reinterpret_cast<void**>(&ex->dev_slots), ex->slot_bytes * slots) ==
                   hipSuccess;
    ok = ok && hipMalloc(reinterpret_cast<void**>(&ex->dev_index),
                         sizeof(int32_t) * 2 * L * E) == hipSuccess;
    ok = ok && hipHostMalloc(reinterpret_cast<void**>(&ex->host_index),
                             sizeof(int32_t) * 2 * L * E, hipHostMallocDefault) == hipSuccess;
    ex->ready.assign(L, nullptr);
    ex->done.assign(L, nullptr);
    for (int32_t l = 0; ok && l < L; ++l) {
        ok = hipEventCreateWithFlags(&ex->ready[l], hipEventDisableTiming) == hipSuccess &&
             hipEventCreateWithFlags(&ex->done[l], hipEventDisableTiming) == hipSuccess;
        // Recorded once so that every later wait refers to a recorded event.
        ok = ok && hipEventRecord(ex->done[l], s) == hipSuccess;
    }
    for (int p = 0; ok && p < 2; ++p)
        ok = hipEventCreateWithFlags(&ex->table_done[p], hipEventDisableTiming) == hipSuccess;
    // Creation is set-up, not the hot path: wait for the host copies here.
    ok = ok && hipStreamSynchronize(s) == hipSuccess;
    if (!ok) {
        release(ex);
        return README_ERR_HIP;
    }
    ex->cache.init(E, L, slots, policy);
    *out = ex;
    return README_OK;
}

void readme_offload_destroy(readme_offload* ex) { release(ex); }

readme_status readme_offload_stats(const readme_offload* ex, int64_t* hits, int64_t* misses,
                                   int64_t* bytes_copied) {
    if (!ex || !hits || !misses || !bytes_copied) return README_ERR_ARG;
    *hits = ex->hits;
    *misses = ex->misses;
    *bytes_copied = ex->bytes;
    return README_OK;
}

readme_status readme_offload_stack(readme_offload* ex, int64_t T, const int32_t* offsets,
                                   const int32_t* counts, const int32_t* next_counts,
                                   float* x_resid_grouped, float rms_eps, void* workspace,
                                   size_t workspace_bytes, void* stream) {
    if (!ex || T < 0 || T > INT32_MAX || !(rms_eps >= 0.0f)) return README_ERR_ARG;
    if (T == 0) return README_OK;
    if (!offsets || !counts || !x_resid_grouped || !workspace) return README_ERR_ARG;
    if (workspace_bytes < readme_moe_ffn_stack_workspace_bytes(T, ex->d, ex->I))
        return README_ERR_WORKSPACE;
    const int E = ex->E, L = ex->L;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);

    for (int e = 0; e < E; ++e)
        if (counts[e] < 0 || (next_counts && next_counts[e] < 0)) return README_ERR_ARG;

    // The slot table buffer of this step's parity was last copied two steps
    // ago; make sure that copy finished before the host rewrites it.
    const int par = (int)(ex->cache.step & 1);
    if (ex->table_used[par] && hipEventSynchronize(ex->table_done[par]) != hipSuccess)
        return README_ERR_HIP;

    // Plan every layer's placement first (it depends only on the references);
    // the planner leaves the cache state unchanged if it fails.
    std::vector<OffloadRef> plan;
    const readme_status pst = offload_plan_step(ex->cache, counts, next_counts, plan);
    if (pst != README_OK) return pst;
    int32_t* table = ex->host_index + (size_t)par * L * E;
    std::fill(table, table + (size_t)L * E, 0);
    struct Copy { int32_t slot, layer, e, wait_layer; };
    std::vector<std::vector<Copy>> copies(L);
    for (const OffloadRef& r : plan) {
        table[(size_t)r.layer * E + r.expert] = r.slot;
        if (r.hit) {
            ++ex->hits;
        } else {
            ++ex->misses;
            ex->bytes += (int64_t)ex->slot_bytes;
            copies[r.layer].push_back({r.slot, r.layer, r.expert, r.wait_layer});
        }
    }
    ex->last_plan = plan;

    auto issue = [&](int l) -> bool {
        for (const Copy& c : copies[l]) {
            if (c.wait_layer >= 0 && hipStreamWaitEvent(ex->copy, ex->done[c.wait_layer], 0) !=
                                         hipSuccess)
                return false;
            char* dst = ex->dev_slots + (size_t)c.slot * ex->slot_bytes;
            const char* src = ex->host[c.layer];
            if (hipMemcpyAsync(dst, src + (size_t)c.e * ex->gu_bytes, ex->gu_bytes,
                               hipMemcpyHostToDevice, ex->copy) != hipSuccess ||
                hipMemcpyAsync(dst + ex->gu_bytes,
                               src + (size_t)E * ex->gu_bytes + (size_t)c.e * ex->dn_bytes,
                               ex->dn_bytes, hipMemcpyHostToDevice, ex->copy) != hipSuccess)
                return false;
        }
        return hipEventRecord(ex->ready[l], ex->copy) == hipSuccess;
    };

    // A failure past this point leaves copies unissued for keys the plan
    // already counts as cached: forget every key, so no later step hits on a
    // slot whose copy never ran.
    auto fail = [&]() {
        ex->cache.clear();
        return README_ERR_HIP;
    };
    int32_t* dev_table = ex->dev_index + (size_t)par * L * E;
    // The copy stream starts after the work already on the compute stream.
    hipEvent_t start = ex->done[L - 1];
    if (hipEventRecord(start, s) != hipSuccess || hipStreamWaitEvent(ex->copy, start, 0) != hipSuccess ||
        hipMemcpyAsync(dev_table, table, sizeof(int32_t) * L * E, hipMemcpyHostToDevice,
                       ex->copy) != hipSuccess ||
        hipEventRecord(ex->table_done[par], ex->copy) != hipSuccess)
        return fail();
    ex->table_used[par] = true;
    if (!issue(0)) return fail();

    uint16_t* xn = reinterpret_cast<uint16_t*>(workspace);
    uint16_t* h = xn + T * ex->d;
    int m32 = 0;  // 32-row tiles of the batch, for the tile choice
    for (int e = 0; e < E; ++e) m32 += (counts[e] + 31) / 32;
    const int64_t slot_elems = (int64_t)(ex->slot_bytes / 2);
    for (int l = 0; l < L; ++l) {
        if (l + 1 < L && !issue(l + 1)) return fail();
        if (hipStreamWaitEvent(s, ex->ready[l], 0) != hipSuccess) return fail();
        hipError_t err = launch_rms_to_bf16(T, ex->d, x_resid_grouped, offsets, E, rms_eps, xn, s);
        GemmArgs gu = gate_up_args(README_BF16, T, ex->d, E, ex->I, xn, offsets, ex->dev_slots, h);
        gu.b_expert_stride = slot_elems;
        gu.b_index = dev_table + (size_t)l * E;
        gu.m_tiles32 = m32;
        if (err == hipSuccess) err = launch_grouped_gemm(false, EPI_GATE_UP_SILU, gu, s);
        GemmArgs dn = down_args(README_BF16, T, ex->d, E, ex->I, h, offsets, ex->dev_slots,
                                x_resid_grouped);
        dn.B = ex->dev_slots + ex->gu_bytes;
        dn.b_expert_stride = slot_elems;
        dn.b_index = dev_table + (size_t)l * E;
        dn.m_tiles32 = m32;
        if (err == hipSuccess) err = launch_grouped_gemm(false, EPI_RESID_ADD, dn, s);
        if (err != hipSuccess || hipEventRecord(ex->done[l], s) != hipSuccess) return fail();
    }
    return README_OK;
}

readme_status readme_offload_last_plan(const readme_offload* ex, int64_t max_refs,
                                       uint8_t* hits, int32_t* slot, int32_t* evicted,
                                       int64_t* n_refs) {
    if (!ex || max_refs < 0 || !n_refs) return README_ERR_ARG;
    const int64_t n = (int64_t)ex->last_plan.size();
    *n_refs = n;
    if (n > max_refs) return README_ERR_WORKSPACE;
    if (n > 0 && (!hits || !slot || !evicted)) return README_ERR_ARG;
    for (int64_t i = 0; i < n; ++i) {
        const OffloadRef& r = ex->last_plan[i];
        hits[i] = r.hit ? 1 : 0;
        slot[i] = r.slot;
        evicted[i] = r.evicted;
    }
    return README_OK;
}

}  // extern "C"
