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
// the copy stream waits on done[] of the slot's last layer.  Keys of the
// layer about to be computed and of the one being loaded are never evicted,
// so a slot is never overwritten while a kernel enqueued before the copy
// may still read it.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <limits>
#include <unordered_map>
#include <vector>

#include "common.hpp"
#include "internal.hpp"

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
    std::vector<int32_t> slot_key;   // key l*E+e held by a slot, -1 empty
    std::vector<int32_t> slot_layer; // layer of the slot's last compute use, -1 none
    std::vector<int64_t> slot_step;  // step of that use
    std::unordered_map<int32_t, int32_t> where;  // key -> slot
    std::unordered_map<int32_t, int64_t> last_ref;  // LRU: key -> reference time
    int64_t clock = 0;
    int64_t step = 0;
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
    ex->slot_key.assign(slots, -1);
    ex->slot_layer.assign(slots, -1);
    ex->slot_step.assign(slots, -1);
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

    // References of this step in layer order (then the next step's, for the
    // Belady look-ahead).
    std::vector<int32_t> active, next_active;
    for (int e = 0; e < E; ++e) {
        if (counts[e] < 0) return README_ERR_ARG;
        if (counts[e] > 0) active.push_back(e);
        if (next_counts && next_counts[e] > 0) next_active.push_back(e);
    }
    // Two layers' experts (the one being loaded and the one computed before
    // it) must fit in the cache at once.
    const int A = (int)active.size();
    if (2 * A > ex->slots) return README_ERR_UNSUPPORTED;
    std::vector<int32_t> refs;
    for (int l = 0; l < L; ++l)
        for (int e : active) refs.push_back(l * E + e);
    for (int l = 0; l < L; ++l)
        for (int e : next_active) refs.push_back(l * E + e);
    const int64_t NEVER = std::numeric_limits<int64_t>::max();
    std::unordered_map<int32_t, std::vector<int64_t>> uses;  // key -> positions, ascending
    for (int64_t t = 0; t < (int64_t)refs.size(); ++t) uses[refs[t]].push_back(t);
    auto next_use = [&](int32_t key, int64_t after) {
        auto it = uses.find(key);
        if (it == uses.end()) return NEVER;
        auto p = std::upper_bound(it->second.begin(), it->second.end(), after);
        return p == it->second.end() ? NEVER : *p;
    };

    // The slot table buffer of this step's parity was last copied two steps
    // ago; make sure that copy finished before the host rewrites it.
    const int par = (int)(ex->step & 1);
    if (ex->table_used[par] && hipEventSynchronize(ex->table_done[par]) != hipSuccess)
        return README_ERR_HIP;
    int32_t* table = ex->host_index + (size_t)par * L * E;
    std::fill(table, table + (size_t)L * E, 0);

    // Plan every layer's placement first (it depends only on the references).
    struct Copy { int32_t slot, layer, e, wait_layer; };
    std::vector<std::vector<Copy>> copies(L);
    int64_t pos = 0;
    for (int l = 0; l < L; ++l) {
        for (int e : active) {
            const int32_t key = l * E + e;
            ++ex->clock;
            auto it = ex->where.find(key);
            int32_t slot;
            if (it != ex->where.end()) {
                slot = it->second;
                ++ex->hits;
            } else {
                ++ex->misses;
                slot = -1;
                for (int32_t q = 0; q < ex->slots && slot < 0; ++q)
                    if (ex->slot_key[q] < 0) slot = q;
                if (slot < 0) {
                    // Victim among keys not of layer l (being placed) nor
                    // used at layer l-1 of this step (its compute is
                    // enqueued after these copies).
                    int64_t best = -1;
                    int32_t best_key = 0;
                    for (int32_t q = 0; q < ex->slots; ++q) {
                        const int32_t k = ex->slot_key[q];
                        const bool now = ex->slot_step[q] == ex->step;
                        if (k / E == l || (now && ex->slot_layer[q] == l - 1)) continue;
                        int64_t v;
                        if (ex->policy == README_CACHE_BELADY)
                            v = next_use(k, pos);                     // farthest next use
                        else
                            v = NEVER - ex->last_ref[k];              // least recent
                        if (v > best || (v == best && k < best_key)) {
                            best = v;
                            best_key = k;
                            slot = q;
                        }
                    }
                    if (slot < 0) return README_ERR_UNSUPPORTED;  // cache too small
                    ex->where.erase(ex->slot_key[slot]);
                }
                copies[l].push_back({slot, l, e, ex->slot_layer[slot]});
                ex->slot_key[slot] = key;
                ex->where[key] = slot;
                ex->bytes += (int64_t)ex->slot_bytes;
            }
            ex->slot_layer[slot] = l;
            ex->slot_step[slot] = ex->step;
            ex->last_ref[key] = ex->clock;
            table[(size_t)l * E + e] = slot;
            ++pos;
        }
    }

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

    int32_t* dev_table = ex->dev_index + (size_t)par * L * E;
    // The copy stream starts after the work already on the compute stream.
    hipEvent_t start = ex->done[L - 1];
    if (hipEventRecord(start, s) != hipSuccess || hipStreamWaitEvent(ex->copy, start, 0) != hipSuccess ||
        hipMemcpyAsync(dev_table, table, sizeof(int32_t) * L * E, hipMemcpyHostToDevice,
                       ex->copy) != hipSuccess ||
        hipEventRecord(ex->table_done[par], ex->copy) != hipSuccess)
        return README_ERR_HIP;
    ex->table_used[par] = true;
    if (!issue(0)) return README_ERR_HIP;

    uint16_t* xn = reinterpret_cast<uint16_t*>(workspace);
    uint16_t* h = xn + T * ex->d;
    int m32 = 0;  // 32-row tiles of the batch, for the tile choice
    for (int e = 0; e < E; ++e) m32 += (counts[e] + 31) / 32;
    const int64_t slot_elems = (int64_t)(ex->slot_bytes / 2);
    for (int l = 0; l < L; ++l) {
        if (l + 1 < L && !issue(l + 1)) return README_ERR_HIP;
        if (hipStreamWaitEvent(s, ex->ready[l], 0) != hipSuccess) return README_ERR_HIP;
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
        if (err != hipSuccess || hipEventRecord(ex->done[l], s) != hipSuccess)
            return README_ERR_HIP;
    }
    ++ex->step;
    return README_OK;
}

}  // extern "C"
