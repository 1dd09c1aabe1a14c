// libbsr C entry points: validate on the host, check the device, enqueue kernels.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "bsr_internal.h"
#include "spmm_tiled.h"

namespace bsr {

namespace {

constexpr int kMaxDevices = 64;

struct DeviceInfo {
    std::atomic<int> state{0};  // 0 unknown, 1 gfx950, -1 other architecture
    int cu_count = 0;
    size_t lds_per_block = 0;
};

DeviceInfo g_devices[kMaxDevices];
std::mutex g_device_mutex;
thread_local char g_last_hip_error[256] = "";

int current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return -1;
    return dev;
}

}  // namespace

void set_last_hip_error(const char *msg) {
    std::snprintf(g_last_hip_error, sizeof(g_last_hip_error), "%s", msg ? msg : "");
}

bsr_status ensure_device() {
    int dev = current_device();
    if (dev < 0) {
        set_last_hip_error("hipGetDevice failed");
        return BSR_ERR_HIP;
    }
    if (dev >= kMaxDevices) return BSR_ERR_UNSUPPORTED;
    DeviceInfo &d = g_devices[dev];
    int st = d.state.load(std::memory_order_acquire);
    if (st == 1) return BSR_OK;
    if (st == -1) return BSR_ERR_ARCH;
    std::lock_guard<std::mutex> lock(g_device_mutex);
    st = d.state.load(std::memory_order_relaxed);
    if (st != 0) return st == 1 ? BSR_OK : BSR_ERR_ARCH;
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) {
        set_last_hip_error(hipGetErrorString(e));
        return BSR_ERR_HIP;
    }
    bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    d.cu_count = prop.multiProcessorCount;
    d.lds_per_block = prop.sharedMemPerBlock;
    d.state.store(ok ? 1 : -1, std::memory_order_release);
    return ok ? BSR_OK : BSR_ERR_ARCH;
}

int auto_slices(const int64_t *tiles, int n, int cu_count) {
    // The largest slice count S with every workgroup resident at once: a product of t token
    // tiles launches ceil(t S / 8) workgroups per XCD (its grid is rounded to a multiple of 8
    // and dealt round robin to the 8 XCDs), and an XCD runs one workgroup per CU at a time
    // (the X tile fills most of a CU's LDS).  One more workgroup per XCD than it has CUs
    // would start a second round and nearly double the time.
    const int64_t per_xcd = (cu_count > 0 ? cu_count : 256) / 8;
    int best = 1;
    for (int S = 2; S <= 1024; ++S) {
        int64_t wgs = 0;
        for (int i = 0; i < n; ++i) wgs += (tiles[i] * S + 7) / 8;
        if (wgs > per_xcd) break;
        best = S;
    }
    return best;
}

int device_cu_count() {
    int dev = current_device();
    return (dev >= 0 && dev < kMaxDevices) ? g_devices[dev].cu_count : 0;
}

size_t device_lds_per_block() {
    int dev = current_device();
    return (dev >= 0 && dev < kMaxDevices) ? g_devices[dev].lds_per_block : 0;
}

}  // namespace bsr

extern "C" {

const char *bsr_last_hip_error(void) { return bsr::g_last_hip_error; }

bsr_status bsr_prune_from_dense(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R,
                                int32_t C, int64_t k, int32_t *indptr, int32_t *indices,
                                float *data, int64_t capacity_blocks, void *workspace,
                                size_t ws_bytes, void *stream) {
    bsr_status s = bsr::check_prune(W, N, K, ldw, R, C, k, indptr, indices, data,
                                    capacity_blocks, workspace, ws_bytes);
    if (s != BSR_OK) return s;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_prune(W, N, K, ldw, R, C, k, indptr, indices, data, workspace,
                             BSR_NORM_L2, BSR_SELECT_GLOBAL, stream);
}

bsr_status bsr_prune_from_dense_noalloc(const float *W, int64_t N, int64_t K, int64_t ldw,
                                        int32_t R, int32_t C, int64_t k, int32_t *indptr,
                                        int32_t *indices, float *data, int64_t capacity_blocks,
                                        void *stream) {
    bsr_status s = bsr::check_prune_noalloc(W, N, K, ldw, R, C, k, indptr, indices, data,
                                            capacity_blocks);
    if (s != BSR_OK) return s;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    void *scratch = nullptr;
    if ((s = bsr::noalloc_scratch(&scratch)) != BSR_OK) return s;
    return bsr::launch_prune(W, N, K, ldw, R, C, k, indptr, indices, data, scratch,
                             BSR_NORM_L2, BSR_SELECT_GLOBAL, stream);
}

bsr_status bsr_prune_from_dense_ex(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R,
                                   int32_t C, int64_t k, int32_t *indptr, int32_t *indices,
                                   float *data, int64_t capacity_blocks, void *workspace,
                                   size_t ws_bytes, const bsr_prune_options_t *opts,
                                   void *stream) {
    bsr_status s = bsr::check_prune(W, N, K, ldw, R, C, k, indptr, indices, data,
                                    capacity_blocks, workspace, ws_bytes);
    if (s != BSR_OK) return s;
    if ((s = bsr::check_prune_options(opts, N, R, k)) != BSR_OK) return s;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_prune(W, N, K, ldw, R, C, k, indptr, indices, data, workspace,
                             opts ? opts->norm : BSR_NORM_L2,
                             opts ? opts->select : BSR_SELECT_GLOBAL, stream);
}

bsr_status bsr_spmm_ex(const void *X, bsr_dtype x_dtype, int64_t T, int64_t ldx,
                       const bsr_matrix_t *W, const float *bias, float *Y, int64_t ldy,
                       const bsr_spmm_options_t *opts, void *stream) {
    bsr_spmm_item_t item{X, BSR_F32, T, ldx, W, bias, Y, ldy};
    memcpy(&item.x_dtype, &x_dtype, sizeof item.x_dtype);   // any int32 the caller passed
    return bsr_spmm_batched(&item, 1, opts, stream);
}

bsr_status bsr_spmm_batched(const bsr_spmm_item_t *items, int32_t n_items,
                            const bsr_spmm_options_t *opts, void *stream) {
    return bsr_spmm_batched_planned(items, nullptr, n_items, opts, stream);
}

bsr_status bsr_plan_bytes_ex(const bsr_matrix_t *W, int32_t arith, size_t *bytes) {
    if (!W || !bytes) return BSR_ERR_NULL;
    bsr_status s = bsr::check_matrix(W);
    if (s != BSR_OK) return s;
    if (bsr::resolve_arith(W->dtype, arith) < 0) return BSR_ERR_ARG;
    const bsr::PlanLayout L = bsr::plan_layout(W, arith);
    if (L.unit_blocks == 0 || L.max_units * 64 >= (int64_t(1) << 31)) return BSR_ERR_UNSUPPORTED;
    *bytes = size_t(L.total);
    return BSR_OK;
}

bsr_status bsr_plan_bytes(const bsr_matrix_t *W, size_t *bytes) {
    return bsr_plan_bytes_ex(W, BSR_ARITH_AUTO, bytes);
}

bsr_status bsr_plan_prepare_ex(const bsr_matrix_t *W, int32_t arith, void *mem, size_t bytes,
                               bsr_plan_t *plan, void *stream) {
    size_t need = 0;
    bsr_status s = bsr_plan_bytes_ex(W, arith, &need);
    if (s != BSR_OK) return s;
    if (!plan) return BSR_ERR_NULL;
    const bsr::PlanLayout L = bsr::plan_layout(W, arith);
    if ((s = bsr::check_plan_prepare(W, mem, bytes, L.total)) != BSR_OK) return s;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    if ((s = bsr::launch_plan_prepare(W, mem, L, stream)) != BSR_OK) return s;
    bsr_plan_t p{};
    p.mem = mem;
    p.bytes = bytes;
    p.n_rows = W->n_rows;
    p.n_cols = W->n_cols;
    p.nnzb = W->nnzb;
    p.R = W->R;
    p.C = W->C;
    p.dtype = int32_t(W->dtype);
    p.indptr = W->indptr;
    p.indices = W->indices;
    p.data = W->data;
    p.unit_blocks = L.unit_blocks;
    p.max_units = L.max_units;
    p.uptr_offset = L.uptr_offset;
    p.col_offset = L.col_offset;
    p.val_offset = L.val_offset;
    p.arith = L.arith;
    *plan = p;
    return BSR_OK;
}

bsr_status bsr_plan_prepare(const bsr_matrix_t *W, void *mem, size_t bytes, bsr_plan_t *plan,
                            void *stream) {
    return bsr_plan_prepare_ex(W, BSR_ARITH_AUTO, mem, bytes, plan, stream);
}

bsr_status bsr_spmm_batched_planned(const bsr_spmm_item_t *items, const bsr_plan_t *const *plans,
                                    int32_t n_items, const bsr_spmm_options_t *opts,
                                    void *stream) {
    if (n_items < 0) return BSR_ERR_ARG;
    if (n_items > 0 && !items) return BSR_ERR_NULL;
    for (int32_t i = 0; i < n_items; ++i) {
        const bsr_spmm_item_t &it = items[i];
        bsr_status s =
            bsr::check_spmm(it.X, bsr::raw_enum(it.x_dtype), it.T, it.ldx, it.W, it.Y, it.ldy,
                            it.bias);
        if (s != BSR_OK) return s;
        const bsr_plan_t *pl = plans ? plans[i] : nullptr;
        if (pl) {
            // The plan's recorded arithmetic must name one (a plan struct filled by hand may
            // hold anything) and its layout must be the one bsr_plan_prepare_ex writes.
            if (pl->arith != BSR_ARITH_NATIVE && pl->arith != BSR_ARITH_BF16X3) return BSR_ERR_ARG;
            const bsr::PlanLayout L = bsr::plan_layout(it.W, pl->arith);
            if (L.unit_blocks == 0 || pl->unit_blocks != L.unit_blocks ||
                pl->max_units != L.max_units || pl->uptr_offset != L.uptr_offset ||
                pl->col_offset != L.col_offset || pl->val_offset != L.val_offset)
                return BSR_ERR_ARG;
            if ((s = bsr::check_plan_use(it, pl, L.total)) != BSR_OK) return s;
        }
    }
    if (n_items > 1) {
        bsr_status s = bsr::check_spmm_items(items, n_items);
        if (s != BSR_OK) return s;
    }
    const int kernel = opts ? opts->kernel : BSR_KERNEL_AUTO;
    const int slices = opts ? opts->slices : 0;
    bsr::LaunchEvents ev;
    if (opts) {
        ev.start = opts->start_event;
        ev.stop = opts->stop_event;
    }
    if (kernel < BSR_KERNEL_AUTO || kernel > BSR_KERNEL_VALU || slices < 0) return BSR_ERR_ARG;
    if ((ev.start == nullptr) != (ev.stop == nullptr)) return BSR_ERR_ARG;

    // Plan: every non-empty product goes to the matrix-core tiled kernel when it has the shape,
    // or, when its X tile is too wide for LDS, to the column-chunked matrix-core kernel; else to
    // the vector-ALU tile kernel or its column-chunked form; else to the generic kernel (a
    // forced kernel choice narrows this; a forced kernel that does not fit is an error).
    enum Kind { kGeneric = 0, kTiled = 1, kVtile = 2, kKchunk = 3, kVchunk = 4, kFlat = 5 };
    std::vector<int> work;
    for (int32_t i = 0; i < n_items; ++i)
        if (items[i].T > 0) work.push_back(i);
    if (work.empty()) return BSR_OK;
    bsr_status s = bsr::ensure_device();
    if (s != BSR_OK) return s;
    const int cus = bsr::device_cu_count();
    const size_t lds_limit = bsr::device_lds_per_block();
    std::vector<bsr::TiledWork> tiled(work.size());
    std::vector<bsr::KchunkWork> kchunk(work.size());
    std::vector<int> kind(work.size(), kGeneric);
    std::vector<int> tokens(work.size(), 32);   // tokens per tile of a flat or tiled launch
    for (size_t w = 0; w < work.size(); ++w) {
        const bsr_spmm_item_t &it = items[work[w]];
        const int R = it.W->R, C = it.W->C, dt = it.W->dtype;
        // A trial plan with one slice decides whether the shape fits.
        if ((kernel == BSR_KERNEL_AUTO || kernel == BSR_KERNEL_TILED) &&
            bsr::tiled_supported(R, C, dt) &&
            bsr::plan_tiled(it.X, it.T, it.ldx, it.W, it.ldy, 1, lds_limit).ok)
            kind[w] = kTiled;
        else if ((kernel == BSR_KERNEL_AUTO || kernel == BSR_KERNEL_TILED) &&
                 bsr::tiled_supported(R, C, dt) &&
                 bsr::plan_kchunk(it.X, it.T, it.ldx, it.W, it.ldy, 1, lds_limit).base.ok)
            kind[w] = kKchunk;
        else if ((kernel == BSR_KERNEL_AUTO || kernel == BSR_KERNEL_VALU) &&
                 bsr::vtile_supported(R, C, dt) &&
                 bsr::plan_vtile(it.X, it.T, it.ldx, it.W, it.ldy, 1, lds_limit).ok)
            kind[w] = kVtile;
        else if ((kernel == BSR_KERNEL_AUTO || kernel == BSR_KERNEL_VALU) &&
                 bsr::vtile_supported(R, C, dt) &&
                 bsr::plan_vchunk(it.X, it.T, it.ldx, it.W, it.ldy, 1, lds_limit).base.ok)
            kind[w] = kVchunk;
        if (kind[w] == kGeneric && (kernel == BSR_KERNEL_TILED || kernel == BSR_KERNEL_VALU))
            return BSR_ERR_UNSUPPORTED;
        // Linear R x 1 blocks run on the flat-stream form of the matrix-core kernel, with the
        // token tile its plan picks (the tiled kernel proper takes 32-token tiles).
        if (kind[w] == kTiled && bsr::flat_supported(R, C, dt)) {
            kind[w] = kFlat;
            tokens[w] = bsr::plan_tiled(it.X, it.T, it.ldx, it.W, it.ldy, 1, lds_limit).tokens;
        }
    }
    // A plan is used where its product runs on the flat kernel (elsewhere it is not needed:
    // the result is the same without it).
    std::vector<const bsr_plan_t *> plan_of(work.size(), nullptr);
    for (size_t w = 0; w < work.size(); ++w)
        if (plans && kind[w] == kFlat) plan_of[w] = plans[work[w]];
    // Launch order: tiled and vector-ALU products grouped by kernel, block shape and dtype, up
    // to kMaxItems per launch, then generic products one by one.  With an event pair, the start
    // event goes with the first launch and the stop event with the last.
    struct Launch {
        int kind;
        std::vector<int> members;  // indices into `work`
    };
    std::vector<Launch> launches;
    std::vector<char> done(work.size(), 0);
    for (size_t w = 0; w < work.size(); ++w) {
        if (kind[w] == kGeneric || done[w]) continue;
        Launch l{kind[w], {}};
        for (size_t v = w; v < work.size(); ++v) {
            if (kind[v] != kind[w] || done[v]) continue;
            if (items[work[v]].W->R != items[work[w]].W->R ||
                items[work[v]].W->C != items[work[w]].W->C ||
                items[work[v]].W->dtype != items[work[w]].W->dtype ||
                (plan_of[v] != nullptr) != (plan_of[w] != nullptr) ||
                (plan_of[v] && plan_of[v]->arith != plan_of[w]->arith) ||
                tokens[v] != tokens[w])
                continue;
            l.members.push_back(int(v));
            done[v] = 1;
            if (int(l.members.size()) == bsr::kMaxItems) {
                launches.push_back(l);
                l.members.clear();
            }
        }
        if (!l.members.empty()) launches.push_back(l);
    }
    for (size_t w = 0; w < work.size(); ++w)
        if (kind[w] == kGeneric) launches.push_back(Launch{kGeneric, {int(w)}});

    // Slices per launch: the automatic count is chosen for the token tiles of the products
    // that share the launch (launches run one after another).
    for (const Launch &l : launches) {
        if (l.kind == kGeneric) continue;
        std::vector<int64_t> tiles;
        for (int w : l.members)
            tiles.push_back((items[work[w]].T + tokens[w] - 1) / tokens[w]);
        const int auto_S = bsr::auto_slices(tiles.data(), int(tiles.size()), cus);
        for (int w : l.members) {
            const bsr_spmm_item_t &it = items[work[w]];
            const int64_t Nb = it.W->n_rows / it.W->R;
            const int S = slices > 0 ? slices : int(auto_S < Nb ? auto_S : Nb);
            if (kind[w] == kKchunk || kind[w] == kVchunk) {
                const bsr::KchunkPlan kp =
                    kind[w] == kKchunk
                        ? bsr::plan_kchunk(it.X, it.T, it.ldx, it.W, it.ldy, S, lds_limit)
                        : bsr::plan_vchunk(it.X, it.T, it.ldx, it.W, it.ldy, S, lds_limit);
                kchunk[w] = bsr::KchunkWork{kp, it.X, it.T, it.ldx, it.W, it.bias, it.Y, it.ldy};
                continue;
            }
            const bsr::TiledPlan plan =
                kind[w] == kVtile
                    ? bsr::plan_vtile(it.X, it.T, it.ldx, it.W, it.ldy, S, lds_limit)
                    : bsr::plan_tiled(it.X, it.T, it.ldx, it.W, it.ldy, S, lds_limit);
            tiled[w] = bsr::TiledWork{plan, it.X, it.T, it.ldx, it.W, it.bias, it.Y, it.ldy};
            if (const bsr_plan_t *pl = plan_of[w]) {
                tiled[w].plan_mem = pl->mem;
                tiled[w].plan_uptr_offset = pl->uptr_offset;
                tiled[w].plan_col_offset = pl->col_offset;
                tiled[w].plan_val_offset = pl->val_offset;
                tiled[w].plan_max_units = pl->max_units;
                tiled[w].plan_arith = pl->arith;
            }
        }
    }

    for (size_t li = 0; li < launches.size(); ++li) {
        bsr::LaunchEvents lev;
        if (li == 0) lev.start = ev.start;
        if (li + 1 == launches.size()) lev.stop = ev.stop;
        const Launch &l = launches[li];
        if (l.kind == kKchunk || l.kind == kVchunk) {
            bsr::KchunkWork batch[bsr::kMaxItems];
            for (size_t m = 0; m < l.members.size(); ++m) batch[m] = kchunk[l.members[m]];
            s = l.kind == kKchunk
                    ? bsr::launch_spmm_kchunk(batch, int(l.members.size()), stream, lev)
                    : bsr::launch_spmm_vchunk(batch, int(l.members.size()), stream, lev);
        } else if (l.kind != kGeneric) {
            bsr::TiledWork batch[bsr::kMaxItems];
            for (size_t m = 0; m < l.members.size(); ++m) batch[m] = tiled[l.members[m]];
            const int nm = int(l.members.size());
            if (l.kind == kFlat)
                s = bsr::launch_spmm_flat(batch, nm, plan_of[l.members[0]] != nullptr, stream, lev);
            else if (l.kind == kTiled)
                s = bsr::launch_spmm_tiled(batch, nm, stream, lev);
            else
                s = bsr::launch_spmm_vtile(batch, nm, stream, lev);
        } else {
            const bsr_spmm_item_t &it = items[work[l.members[0]]];
            s = bsr::launch_spmm_generic(it.X, it.T, it.ldx, it.W, it.bias, it.Y, it.ldy, stream,
                                         lev);
        }
        if (s != BSR_OK) return s;
    }
    return BSR_OK;
}

bsr_status bsr_spmm(const void *X, bsr_dtype x_dtype, int64_t T, int64_t ldx,
                    const bsr_matrix_t *W, const float *bias, float *Y, int64_t ldy,
                    void *stream) {
    return bsr_spmm_ex(X, x_dtype, T, ldx, W, bias, Y, ldy, nullptr, stream);
}

bsr_status bsr_to_dense(const bsr_matrix_t *W, float *out, int64_t ldo, void *stream) {
    bsr_status s = bsr::check_to_dense(W, out, ldo);
    if (s != BSR_OK) return s;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_to_dense(W, out, ldo, stream);
}

bsr_status bsr_attention(const float *Q, int64_t ldq, const float *K, int64_t ldk,
                         const float *V, int64_t ldv, float *O, int64_t ldo, int32_t batch,
                         int32_t seq, int32_t heads, int32_t head_dim, float scale,
                         void *stream) {
    bsr_status s = bsr::check_attention(Q, ldq, K, ldk, V, ldv, O, ldo, batch, seq, heads,
                                        head_dim, scale);
    if (s != BSR_OK) return s;
    if (int64_t(batch) * seq == 0) return BSR_OK;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_attention(Q, ldq, K, ldk, V, ldv, O, ldo, batch, seq, heads, scale,
                                 stream);
}

bsr_status bsr_reblock(const bsr_matrix_t *W, int32_t R2, int32_t C2, int32_t *indptr_out,
                       int32_t *indices_out, void *data_out, void *stream) {
    bsr_status s = bsr::check_reblock(W, R2, C2, indptr_out, indices_out, data_out);
    if (s != BSR_OK) return s;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_reblock(W, R2, C2, indptr_out, indices_out, data_out, stream);
}

bsr_status bsr_iht_update(const float *W, int64_t ldw, const float *G, int64_t ldg,
                          const float *C0, int64_t ldc, float eta, int64_t N, int64_t K, float *V,
                          int64_t ldv, void *stream) {
    bsr_status s = bsr::check_iht_update(W, ldw, G, ldg, C0, ldc, eta, N, K, V, ldv);
    if (s != BSR_OK) return s;
    if (N == 0 || K == 0) return BSR_OK;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_iht_update(W, ldw, G, ldg, C0, ldc, eta, N, K, V, ldv, stream);
}

bsr_status bsr_cast_f32_bf16(const float *src, uint16_t *dst, int64_t n, void *stream) {
    bsr_status s = bsr::check_cast(src, dst, n);
    if (s != BSR_OK) return s;
    if (n == 0) return BSR_OK;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_cast(src, dst, n, stream);
}

}  // extern "C"
