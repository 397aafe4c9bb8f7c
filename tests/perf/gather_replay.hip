// Gather ceilings for the PatchMatch sweep (a measurement aid, not part of the library).
//
//   gather_replay DIR TAG   replays the row lists DIR/rows_TAG.bin, DIR/cnt_TAG.bin written by
//                           sweep_rows.py: one lane group of 4 lanes per query (as the sweep
//                           kernel), which reads its own query row and then its key rows -- the
//                           first ones in batches of 4, the last RS one after another, each
//                           address depending on the previous row (as random search does) --
//                           and does no arithmetic beyond folding the data into a checksum.
//   gather_replay --random N  each lane group reads 32 rows drawn uniformly from the first N
//                           rows of an 8 MiB table, for 4 and 8 lanes per row.
//
// Tables are bf16 rows of d = 64 (128 bytes); 4 slices of 65536 keys.  Every launch is timed
// after 400 warm-up launches, averaged over 200.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <string_view>
#include <vector>

#define CHECK(x)                                                                  \
    do {                                                                          \
        hipError_t e_ = (x);                                                      \
        if (e_ != hipSuccess) {                                                   \
            std::printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            return 1;                                                             \
        }                                                                         \
    } while (0)

namespace {

constexpr int kSlices = 4, kKeys = 65536, kD = 64, kMaxRows = 32, kRs = 8, kRandomRows = 32;

// the sweep kernel's block order: XCD x (blocks x, x + 8, ...) takes the x-th contiguous eighth
__device__ uint32_t xcd_order(uint32_t b, uint32_t nb)
{
    const uint32_t x = b % 8, local = b / 8, q = nb / 8, r = nb % 8;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + local;
}

__global__ __launch_bounds__(256) void replay(const uint4* __restrict__ Q, const uint4* __restrict__ K,
                                              const int* __restrict__ rows, const int* __restrict__ cnt,
                                              uint32_t zero, uint32_t* sink)
{
    const int lane = threadIdx.x & 3;
    const uint32_t g = xcd_order(blockIdx.x, gridDim.x) * 64 + threadIdx.x / 4;
    if (g >= static_cast<uint32_t>(kSlices * kKeys)) return;
    const uint4* Ks = K + static_cast<size_t>(g / kKeys) * kKeys * 8;
    const uint4 q0 = Q[static_cast<size_t>(g) * 8 + lane], q1 = Q[static_cast<size_t>(g) * 8 + lane + 4];
    uint32_t acc = q0.x ^ q0.y ^ q0.z ^ q0.w ^ q1.x ^ q1.y ^ q1.z ^ q1.w;
    const int n = cnt[g];
    const int* my = rows + static_cast<size_t>(g) * kMaxRows;
    const int4* my4 = reinterpret_cast<const int4*>(my);
    const int n1 = n - kRs;
    for (int k0 = 0; k0 < n1; k0 += 4) {
        const int4 v = my4[k0 / 4];
        const int ix[4] = {v.x, v.y, v.z, v.w};
        uint4 a[4], b[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint4* r = Ks + static_cast<size_t>(k0 + e < n1 ? ix[e] : ix[0]) * 8;
            a[e] = r[lane];
            b[e] = r[lane + 4];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
            acc += k0 + e < n1 ? (a[e].x ^ a[e].y ^ a[e].z ^ a[e].w ^ b[e].x ^ b[e].y ^ b[e].z ^ b[e].w) : 0u;
    }
    uint32_t dep = 0;  // zero at run time; the compiler cannot drop the dependency
    for (int k = n1; k < n; ++k) {
        const uint4* r = Ks + static_cast<size_t>(my[k] + dep) * 8;
        const uint4 a = r[lane], b = r[lane + 4];
        acc += a.x ^ a.y ^ b.x ^ b.y;
        dep = (a.z ^ a.w ^ b.z ^ b.w) & zero;
    }
    if (acc == 0x9E3779B9u) sink[0] = acc;
}

template <int G>
__global__ __launch_bounds__(256) void random_rows(const uint4* __restrict__ K, const int* __restrict__ idx,
                                                   int groups, uint32_t* sink)
{
    constexpr int CH = 8 / G;
    const int lane = threadIdx.x & (G - 1);
    const int grp = (blockIdx.x * 256 + threadIdx.x) / G;
    if (grp >= groups) return;
    const int* my = idx + static_cast<size_t>(grp) * kRandomRows;
    uint32_t acc = 0;
#pragma unroll 4
    for (int r = 0; r < kRandomRows; ++r) {
        const uint4* row = K + static_cast<size_t>(my[r]) * 8;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const uint4 v = row[lane + c * G];
            acc ^= v.x + v.y + v.z + v.w;
        }
    }
    if (acc == 0x9E3779B9u) sink[0] = acc;
}

template <typename F>
int time_launches(F&& launch, double* us)
{
    hipEvent_t a, b;
    CHECK(hipEventCreate(&a));
    CHECK(hipEventCreate(&b));
    for (int w = 0; w < 400; ++w) launch();
    CHECK(hipGetLastError());
    CHECK(hipEventRecord(a));
    const int reps = 200;
    for (int w = 0; w < reps; ++w) launch();
    CHECK(hipEventRecord(b));
    CHECK(hipEventSynchronize(b));
    float ms = 0.f;
    CHECK(hipEventElapsedTime(&ms, a, b));
    *us = ms * 1e3 / reps;
    CHECK(hipEventDestroy(a));
    CHECK(hipEventDestroy(b));
    return 0;
}

int read_file(const char* path, void* dst, size_t bytes)
{
    FILE* f = std::fopen(path, "rb");
    if (!f) return 1;
    const size_t got = std::fread(dst, 1, bytes, f);
    std::fclose(f);
    return got == bytes ? 0 : 1;
}

}  // namespace

int main(int argc, char** argv)
{
    if (argc < 3) {
        std::printf("usage: %s DIR TAG | --random N\n", argv[0]);
        return 2;
    }
    const size_t table_rows = static_cast<size_t>(kSlices) * kKeys;
    uint4 *Q, *K;
    uint32_t* sink;
    CHECK(hipMalloc(&Q, table_rows * 128));
    CHECK(hipMalloc(&K, table_rows * 128));
    CHECK(hipMalloc(&sink, 4));
    CHECK(hipMemset(Q, 0x3c, table_rows * 128));
    CHECK(hipMemset(K, 0x3c, table_rows * 128));

    if (std::string_view(argv[1]) == "--random") {
        int spread = std::atoi(argv[2]);
        if (spread < 1 || spread > kKeys) spread = kKeys;
        const int groups = kSlices * kKeys;
        std::vector<int> h(static_cast<size_t>(groups) * kRandomRows);
        std::mt19937 rng(1);
        for (auto& x : h) x = static_cast<int>(rng() % static_cast<uint32_t>(spread));
        int* idx;
        CHECK(hipMalloc(&idx, h.size() * 4));
        CHECK(hipMemcpy(idx, h.data(), h.size() * 4, hipMemcpyHostToDevice));
        const double rows = static_cast<double>(groups) * kRandomRows;
        double us4 = 0, us8 = 0;
        if (time_launches([&] { hipLaunchKernelGGL(random_rows<4>, dim3(groups * 4 / 256), dim3(256), 0, 0, K, idx, groups, sink); }, &us4)) return 1;
        if (time_launches([&] { hipLaunchKernelGGL(random_rows<8>, dim3(groups * 8 / 256), dim3(256), 0, 0, K, idx, groups, sink); }, &us8)) return 1;
        std::printf("uniform rows from %d (%.2f MiB): 4 lanes/row %.1f us = %.1f G rows/s; 8 lanes/row %.1f us = %.1f G rows/s\n",
                    spread, spread * 128.0 / (1 << 20), us4, rows / us4 * 1e-3, us8, rows / us8 * 1e-3);
        CHECK(hipFree(idx));
    } else {
        std::vector<int> rows(table_rows * kMaxRows), cnt(table_rows);
        char path[512];
        std::snprintf(path, sizeof path, "%s/rows_%s.bin", argv[1], argv[2]);
        if (read_file(path, rows.data(), rows.size() * 4)) { std::printf("cannot read %s\n", path); return 1; }
        std::snprintf(path, sizeof path, "%s/cnt_%s.bin", argv[1], argv[2]);
        if (read_file(path, cnt.data(), cnt.size() * 4)) { std::printf("cannot read %s\n", path); return 1; }
        double total = 0;
        for (size_t g = 0; g < cnt.size(); ++g) {  // every index inside its slice's table
            if (cnt[g] < kRs || cnt[g] > kMaxRows) { std::printf("bad count at query %zu\n", g); return 1; }
            for (int k = 0; k < cnt[g]; ++k)
                if (rows[g * kMaxRows + k] < 0 || rows[g * kMaxRows + k] >= kKeys) { std::printf("bad row at query %zu\n", g); return 1; }
            total += cnt[g] + 1;
        }
        int *rd, *cd;
        CHECK(hipMalloc(&rd, rows.size() * 4));
        CHECK(hipMalloc(&cd, cnt.size() * 4));
        CHECK(hipMemcpy(rd, rows.data(), rows.size() * 4, hipMemcpyHostToDevice));
        CHECK(hipMemcpy(cd, cnt.data(), cnt.size() * 4, hipMemcpyHostToDevice));
        double us = 0;
        const uint32_t blocks = static_cast<uint32_t>(table_rows / 64);
        if (time_launches([&] { hipLaunchKernelGGL(replay, dim3(blocks), dim3(256), 0, 0, Q, K, rd, cd, 0u, sink); }, &us)) return 1;
        std::printf("replay %s: %.2f rows per query (own row included): %.1f us per launch = %.1f G rows/s\n",
                    argv[2], total / cnt.size(), us, total / us * 1e-3);
        CHECK(hipFree(rd));
        CHECK(hipFree(cd));
    }
    CHECK(hipDeviceSynchronize());
    CHECK(hipFree(Q));
    CHECK(hipFree(K));
    CHECK(hipFree(sink));
    return 0;
}
