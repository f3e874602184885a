// Measurement tool (not part of the library): the fixed cost of one kernel
// launch and the rate at which one launch can stream a given number of bytes
// from HBM, at the decode-attention kernel's launch shape.  These bound what
// one attention launch per layer can reach, whatever its arithmetic.
//
//   probe_empty   256 blocks of 1024 threads that do nothing: the launch floor
//   probe_read    a balanced read of S bytes: block b streams bytes
//                 [b*S/G, (b+1)*S/G) with 16-byte non-temporal loads, all
//                 loads of a pass issued before use, and writes one sum per
//                 column (every loaded word is used)
//
// Launches rotate over 32 buffers of S bytes, so that (as in a decode step
// over 32 layers) the data is not in the 256 MB Infinity Cache when it is read.
// Usage: stream_probe [MB per launch, default 48] [launches per case, 640].
// For each case it prints the wall time per launch of a back-to-back series
// (events around the series), then the mean duration of each launch of a
// second series from its own start and stop events (hipExtLaunchKernelGGL,
// the kernel's own timestamps, as the library's benchmark times its
// kernels).  Run it under rocprofv3 --kernel-trace --stats for the
// profiler's durations of the same kernels.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

#define CHECK(x)                                                                      \
    do {                                                                              \
        hipError_t e_ = (x);                                                          \
        if (e_ != hipSuccess) {                                                       \
            std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), \
                         __LINE__);                                                   \
            std::exit(1);                                                             \
        }                                                                             \
    } while (0)

template <int T>
__global__ __launch_bounds__(T) void probe_empty(float* out, int flag) {
    if (flag == 12345 && threadIdx.x == 0) out[blockIdx.x] = 1.f;
}

// NL loads per thread and pass; indices past the block's range are clamped to
// its last unit (a repeated address, no extra traffic).
template <int T, int NL>
__global__ __launch_bounds__(T) void probe_read(const u32x4* __restrict__ p, size_t units,
                                                size_t per_block, float* __restrict__ out) {
    const size_t b0 = (size_t)blockIdx.x * per_block;
    const size_t b1 = b0 + per_block < units ? b0 + per_block : units;
    float acc = 0.f;
    for (size_t u0 = b0; u0 < b1; u0 += (size_t)T * NL) {
        u32x4 x[NL];
#pragma unroll
        for (int j = 0; j < NL; ++j) {
            const size_t u = u0 + (size_t)j * T + threadIdx.x;
            x[j] = __builtin_nontemporal_load(p + (u < b1 ? u : b1 - 1));
        }
#pragma unroll
        for (int j = 0; j < NL; ++j)
            acc += __uint_as_float(x[j].x) + __uint_as_float(x[j].y) + __uint_as_float(x[j].z) +
                   __uint_as_float(x[j].w);
    }
    __shared__ float red[T];
    red[threadIdx.x] = acc;
    __syncthreads();
    if (threadIdx.x < 128) {
        float o = 0.f;
        for (int w = 0; w < T / 128; ++w) o += red[threadIdx.x + 128 * w];
        out[(size_t)blockIdx.x * 128 + threadIdx.x] = o;
    }
}

int main(int argc, char** argv) {
    const size_t mb = argc > 1 ? std::strtoull(argv[1], nullptr, 10) : 48;
    const int n = argc > 2 ? std::atoi(argv[2]) : 640;
    if (mb < 1 || mb > 1024 || n < 1 || n > 100000) {
        std::fprintf(stderr, "usage: stream_probe [MB 1..1024] [launches 1..100000]\n");
        return 2;
    }
    const int L = 32;
    const size_t big = 2 * (mb << 20);  // the largest case reads twice the size
    std::vector<u32x4*> buf(L);
    for (int l = 0; l < L; ++l) {
        CHECK(hipMalloc(&buf[l], big));
        CHECK(hipMemset(buf[l], 0, big));
    }
    float* out;
    const int max_blocks = 2048;
    CHECK(hipMalloc(&out, (size_t)max_blocks * 128 * sizeof(float)));
    hipEvent_t a, b;
    CHECK(hipEventCreate(&a));
    CHECK(hipEventCreate(&b));
    std::vector<hipEvent_t> e0(n), e1(n);
    for (int i = 0; i < n; ++i) {
        CHECK(hipEventCreate(&e0[i]));
        CHECK(hipEventCreate(&e1[i]));
    }
    // launch(i, start, stop): null events for a plain launch
    auto series = [&](const char* name, auto launch) {
        for (int i = 0; i < 64; ++i) launch(i, nullptr, nullptr);  // warm-up
        CHECK(hipDeviceSynchronize());
        CHECK(hipEventRecord(a, nullptr));
        for (int i = 0; i < n; ++i) launch(i, nullptr, nullptr);
        CHECK(hipEventRecord(b, nullptr));
        CHECK(hipEventSynchronize(b));
        CHECK(hipGetLastError());
        float ms = 0.f;
        CHECK(hipEventElapsedTime(&ms, a, b));
        for (int i = 0; i < n; ++i) launch(i, e0[i], e1[i]);
        CHECK(hipDeviceSynchronize());
        CHECK(hipGetLastError());
        double own = 0.0;
        for (int i = 0; i < n; ++i) {
            float t = 0.f;
            CHECK(hipEventElapsedTime(&t, e0[i], e1[i]));
            own += t;
        }
        std::printf("%-44s %8.2f us per launch back to back, %8.2f us per launch from its own events\n",
                    name, ms * 1e3 / n, own * 1e3 / n);
        std::fflush(stdout);
    };
    series("empty, 256 x 1024 threads", [&](int, hipEvent_t s0, hipEvent_t s1) {
        hipExtLaunchKernelGGL(probe_empty<1024>, dim3(256), dim3(1024), 0, nullptr, s0, s1, 0,
                              out, 0);
    });
    for (size_t bytes : {mb << 20, 2 * (mb << 20)}) {
        const size_t units = bytes / 16;
        char name[96];
        const size_t pb1 = (units + 255) / 256;
        std::snprintf(name, sizeof name, "read %zu MB, 256 x 1024 threads", bytes >> 20);
        series(name, [&](int i, hipEvent_t s0, hipEvent_t s1) {
            hipExtLaunchKernelGGL((probe_read<1024, 12>), dim3(256), dim3(1024), 0, nullptr, s0,
                                  s1, 0, buf[i % L], units, pb1, out);
        });
        const size_t pb8 = (units + max_blocks - 1) / max_blocks;
        std::snprintf(name, sizeof name, "read %zu MB, 2048 x 256 threads", bytes >> 20);
        series(name, [&](int i, hipEvent_t s0, hipEvent_t s1) {
            hipExtLaunchKernelGGL((probe_read<256, 12>), dim3(max_blocks), dim3(256), 0, nullptr,
                                  s0, s1, 0, buf[i % L], units, pb8, out);
        });
    }
    for (int i = 0; i < n; ++i) {
        CHECK(hipEventDestroy(e0[i]));
        CHECK(hipEventDestroy(e1[i]));
    }
    for (auto p : buf) CHECK(hipFree(p));
    CHECK(hipFree(out));
    return 0;
}
