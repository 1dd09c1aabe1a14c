// Host-side fuzz of libbsr's argument validation (csrc/validate.cpp), built with AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_host_sanitizers.py.  Every check runs on the host
// only and never dereferences a device pointer, so the pointers here are arbitrary addresses;
// host structs (matrix descriptors, batch items, plans) are real.  The sanitizers flag any
// signed overflow, out-of-range shift or out-of-bounds host access the checks make on hostile
// sizes, pitches and counts.  Prints "ok" and the number of calls when done.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>

#include "bsr_internal.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next() {   // xorshift64*
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return g_state * 0x2545F4914F6CDD1Dull;
}

const int64_t kI64[] = {0, 1, 2, 3, 7, 8, 31, 32, 33, 63, 64, 96, 128, 768, 1000, 1024, 2304, 3072,
                        4096, 6144, (int64_t(1) << 20), (int64_t(1) << 31) - 1, int64_t(1) << 31,
                        int64_t(1) << 32, int64_t(1) << 40, int64_t(1) << 53, (int64_t(1) << 62),
                        std::numeric_limits<int64_t>::max(), -1, -2, -1024,
                        std::numeric_limits<int64_t>::min()};
const int32_t kI32[] = {0, 1, 2, 3, 4, 8, 16, 32, 33, 64, 128, 384, 1024, 65535, 65536,
                        std::numeric_limits<int32_t>::max(), -1, -32,
                        std::numeric_limits<int32_t>::min()};

int64_t i64() {
    if (next() % 4 == 0) return int64_t(next() % 5000) - 100;
    return kI64[next() % (sizeof(kI64) / sizeof(kI64[0]))];
}
int32_t i32() {
    if (next() % 4 == 0) return int32_t(next() % 70) - 2;
    return kI32[next() % (sizeof(kI32) / sizeof(kI32[0]))];
}
const void *ptr() {   // never dereferenced by the checks
    switch (next() % 6) {
        case 0: return nullptr;
        case 1: return reinterpret_cast<const void *>(uintptr_t(0x10000) + (next() % 4096) * 4);
        case 2: return reinterpret_cast<const void *>(uintptr_t(1) << 40);
        case 3: return reinterpret_cast<const void *>(~uintptr_t(0) - 4095);
        case 4: return reinterpret_cast<const void *>(uintptr_t(0x20000) + (next() % 64) * 256);
        default: return reinterpret_cast<const void *>(uintptr_t(0x7f0000000000) + (next() % 1024) * 16);
    }
}
template <class T> const T *p() { return static_cast<const T *>(ptr()); }
int64_t sat_add(int64_t a, int64_t b) {   // b >= 0
    return a > std::numeric_limits<int64_t>::max() - b ? a : a + b;
}
float f32() {
    const float v[] = {0.0f, 1.0f, -1.0f, 0.125f, 1e30f, std::nanf(""),
                       std::numeric_limits<float>::infinity(), 1e-30f};
    return v[next() % 8];
}
double f64() {
    const double v[] = {0.0, 0.1, 0.5, 1.0, -0.1, 1.5, std::nan(""),
                        std::numeric_limits<double>::infinity(), 1e-300};
    return v[next() % 9];
}

// Half of the matrices are well formed (shape tiled by the block, nnzb in range, arrays set),
// so that the checks past the shape tests run too.
bsr_matrix_t valid_matrix() {
    const int32_t shapes[] = {1, 2, 4, 8, 16, 32, 64};
    bsr_matrix_t m{};
    m.R = shapes[next() % 7];
    m.C = shapes[next() % 7];
    const int64_t nbs[] = {1, 2, 3, 24, 32, 72, 1000, int64_t(1) << 20, int64_t(1) << 31};
    const int64_t Nb = nbs[next() % 9], Kb = nbs[next() % 6];
    m.n_rows = Nb * m.R;
    m.n_cols = Kb * m.C;
    m.nnzb = next() % 2 ? 0 : int64_t(next() % uint64_t(Nb * Kb < (int64_t(1) << 31) ? Nb * Kb + 1 : 1000));
    m.dtype = next() % 2 ? BSR_F32 : BSR_BF16;
    m.indptr = reinterpret_cast<const int32_t *>(uintptr_t(0x100000000));
    m.indices = reinterpret_cast<const int32_t *>(uintptr_t(0x200000000));
    m.data = reinterpret_cast<const void *>(uintptr_t(0x300000000));
    return m;
}

bsr_matrix_t matrix() {
    if (next() % 2) return valid_matrix();
    bsr_matrix_t m{};
    m.n_rows = i64();
    m.n_cols = i64();
    m.R = i32();
    m.C = i32();
    m.nnzb = i64();
    m.dtype = bsr_dtype(int32_t(next() % 3) - (next() % 5 == 0 ? 7 : 0));
    m.indptr = p<int32_t>();
    m.indices = p<int32_t>();
    m.data = ptr();
    return m;
}

}  // namespace

int main() {
    long calls = 0, batches = 0;
    volatile int sink = 0;
    for (int it = 0; it < 200000; ++it) {
        switch (it % 12) {
            case 0:
                sink += bsr::check_prune(p<float>(), i64(), i64(), i64(), i32(), i32(), i64(),
                                         p<int32_t>(), p<int32_t>(), p<float>(), i64(), ptr(),
                                         size_t(i64()));
                break;
            case 1:
                sink += bsr::check_prune_noalloc(p<float>(), i64(), i64(), i64(), i32(), i32(),
                                                 i64(), p<int32_t>(), p<int32_t>(), p<float>(),
                                                 i64());
                break;
            case 2: {
                bsr_matrix_t m = matrix();
                sink += bsr::check_matrix(next() % 10 ? &m : nullptr);
                sink += bsr::check_spmm(ptr(), int(next() % 3), i64(), i64(), &m, p<float>(),
                                        i64(), p<float>());
                break;
            }
            case 3: {
                bsr_matrix_t m = matrix();
                sink += bsr::check_to_dense(&m, p<float>(), i64());
                sink += bsr::check_reblock(&m, i32(), i32(), p<int32_t>(), p<int32_t>(), ptr());
                break;
            }
            case 4:
                sink += bsr::check_cast(p<float>(), p<uint16_t>(), i64());
                break;
            case 5:
                sink += bsr::check_attention(p<float>(), i64(), p<float>(), i64(), p<float>(),
                                             i64(), p<float>(), i64(), i32(), i32(), i32(),
                                             i32(), f32());
                break;
            case 6:
                sink += bsr::check_iht_update(p<float>(), i64(), p<float>(), i64(), p<float>(),
                                              i64(), f32(), i64(), i64(), p<float>(), i64());
                break;
            case 7: {
                bsr_prune_options_t o{};
                o.norm = int32_t(next() % 3);
                o.select = int32_t(next() % 3);
                int64_t k = 0;
                // Precondition (as in bsr_prune_from_dense_ex): check_prune passed.
                const int64_t N = i64(), K = i64(), kk = i64();
                const int32_t R = i32(), C = i32();
                if (bsr::check_prune(p<float>(), N, K, K, R, C, kk, p<int32_t>(), p<int32_t>(),
                                     p<float>(), kk, ptr(), ~size_t(0)) == BSR_OK)
                    sink += bsr::check_prune_options(next() % 8 ? &o : nullptr, N, R, kk);
                sink += bsr_prune_count(i64(), i64(), i32(), i32(), f64(),
                                        next() % 10 ? &k : nullptr);
                sink += bsr_prune_count_ex(i64(), i64(), i32(), i32(), f64(),
                                           next() % 4 ? &o : nullptr, next() % 10 ? &k : nullptr);
                sink += int(bsr_prune_workspace_bytes(i64(), i64(), i32(), i32()) & 1);
                break;
            }
            case 8: {   // batches of up to 8 items with aliasing between them
                bsr_matrix_t ms[8];
                bsr_spmm_item_t items[8];
                const int n = int(next() % 9);
                for (int i = 0; i < n; ++i) {
                    ms[i] = matrix();
                    const bool good = next() % 2;
                    items[i].X = good ? reinterpret_cast<const void *>(uintptr_t(0x400000000) +
                                                                       (next() % 4) * 0x10000000)
                                      : ptr();
                    items[i].x_dtype = good ? bsr_dtype(bsr::raw_enum(ms[i].dtype) & 1) : bsr_dtype(next() % 2);
                    items[i].T = good ? int64_t(next() % 300) : i64();
                    items[i].ldx = good ? sat_add(ms[i].n_cols, int64_t(next() % 3)) : i64();
                    items[i].W = &ms[i];
                    items[i].bias = next() % 2 ? nullptr : p<float>();
                    items[i].Y = good ? reinterpret_cast<float *>(uintptr_t(0x500000000) +
                                                                 (next() % 8) * 0x1000000)
                                      : const_cast<float *>(p<float>());
                    items[i].ldy = good ? sat_add(ms[i].n_rows, int64_t(next() % 3)) : i64();
                }
                // Precondition (as in bsr_spmm_batched): every item passed check_spmm.
                bool valid = true;
                for (int i = 0; i < n && valid; ++i)
                    valid = bsr::check_spmm(items[i].X, bsr::raw_enum(items[i].x_dtype),
                                            items[i].T, items[i].ldx, items[i].W, items[i].Y,
                                            items[i].ldy, items[i].bias) == BSR_OK;
                if (valid) {
                    sink += bsr::check_spmm_items(items, n);
                    ++batches;
                }
                break;
            }
            case 9: {   // plans against items
                bsr_matrix_t m = matrix();
                bsr_spmm_item_t item{};
                item.X = ptr();
                item.T = i64();
                item.ldx = i64();
                item.W = &m;
                item.Y = const_cast<float *>(p<float>());
                item.ldy = i64();
                bsr_plan_t plan{};
                plan.mem = const_cast<void *>(ptr());
                plan.bytes = size_t(i64());
                plan.n_rows = next() % 2 ? m.n_rows : i64();
                plan.n_cols = next() % 2 ? m.n_cols : i64();
                plan.nnzb = next() % 2 ? m.nnzb : i64();
                plan.R = next() % 2 ? m.R : i32();
                plan.C = next() % 2 ? m.C : i32();
                plan.dtype = bsr::raw_enum(m.dtype);
                plan.indptr = m.indptr;
                plan.indices = m.indices;
                plan.data = m.data;
                plan.unit_blocks = i32();
                plan.max_units = i64();
                plan.uptr_offset = i64();
                plan.col_offset = i64();
                plan.val_offset = i64();
                // Preconditions: check_spmm passed for the item, check_matrix for the matrix.
                if (bsr::check_spmm(item.X, 0, item.T, item.ldx, &m, item.Y, item.ldy,
                                    nullptr) == BSR_OK)
                    sink += bsr::check_plan_use(item, &plan, i64());
                if (bsr::check_matrix(&m) == BSR_OK)
                    sink += bsr::check_plan_prepare(&m, ptr(), size_t(i64()), i64());
                break;
            }
            case 10:
                for (int s = -2; s < 12; ++s) sink += int(std::strlen(bsr_status_str(bsr_status(s))));
                break;
            default: {
                const int64_t nb = i64();
                if (nb >= 0 && nb < (int64_t(1) << 40)) {
                    bsr::PruneWorkspace w = bsr::prune_workspace_layout(nb);
                    sink += int(w.total & 1);
                }
                break;
            }
        }
        ++calls;
    }
    std::printf("ok %ld calls, %ld batches past check_spmm\n", calls, batches);
    return sink == 12345678 ? 1 : 0;
}
