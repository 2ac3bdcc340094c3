// noalloc.hip -- bytecomp_compress_noalloc: the compress entry point for
// callers that cannot allocate device memory (code under HIP graph capture,
// tight serving loops, harnesses that forbid allocation).  It runs exactly
// the kernels of bytecomp_compress; its workspace and descriptor table live
// in one file-scope device array instead of a caller's workspace and the
// library's descriptor cache, and the descriptor table is written by kernel
// launches (the descriptors travel as kernel arguments), so the call makes
// no allocation and no host-to-device copy.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>

#include "launch.hpp"

namespace bc {

namespace {

// The call's workspace (compress-only plan) followed by its descriptor
// table and chunk -> tensor map.  Each GPU holds its own copy until the
// process ends; every call on a GPU uses it, so calls that overlap on one
// GPU (other streams, other threads) race.
constexpr size_t kScratchBytes = size_t(16) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on each device (the array's name in host code
// is a stand-in, not that address), looked up once per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

hipError_t scratch_address(int dev, unsigned char** out) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!ptr) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = ptr;
    }
    *out = (unsigned char*)g_scratch_ptr[dev];
    return hipSuccess;
}

size_t round256(size_t x) { return (x + 255u) & ~(size_t)255u; }

// Descriptors written by kernel launches: each launch carries up to
// kBlobWords 32-bit words of the table as its argument and stores them.
constexpr int kBlobWords = 768;  // 3072 bytes, well inside the kernel-argument limit
struct Blob {
    uint32_t w[kBlobWords];
};

__global__ void put_words(uint32_t* __restrict__ dst, Blob b, int count) {
    for (int i = threadIdx.x; i < count; i += blockDim.x) dst[i] = b.w[i];
}

// Chunk -> tensor map after the table: chunk c belongs to the last tensor
// whose first chunk is at most c (find_owner).
__global__ void build_chunk_map(const TDesc* __restrict__ d, int T, uint32_t C) {
    uint32_t* map = (uint32_t*)(d + T);
    for (uint32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x)
        map[c] = (uint32_t)find_owner<TDesc, &TDesc::chunk0>(d, T, c);
}

__global__ void zero_words(uint32_t* __restrict__ p, int count) {
    for (int i = threadIdx.x; i < count; i += blockDim.x) p[i] = 0u;
}

}  // namespace

}  // namespace bc

using namespace bc;

extern "C" int bytecomp_compress_noalloc(int kind, double ratio, uint64_t seed, const bc_tensor* t, int T,
                                         bc_payload out, void* stream) {
    const CallRange range("bytecomp_compress_noalloc");
    CompressPrep p;
    int rc = compress_prepare(kind, ratio, t, T, out, false, p);
    if (rc || T == 0) return rc;
    const size_t ws_bytes = round256(p.plan.total);
    const size_t table_bytes = (size_t)T * sizeof(TDesc) + (size_t)p.C * 4u;
    if (ws_bytes + round256(table_bytes) > kScratchBytes) return BC_E_SIZE;
    hipStream_t s = (hipStream_t)stream;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return BC_E_HIP;
    if (dev < 0 || dev >= kMaxDevices) return BC_E_HIP;
    unsigned char* base = nullptr;
    if (scratch_address(dev, &base) != hipSuccess) return BC_E_HIP;
    uint32_t* ws = (uint32_t*)base;
    TDesc* dd = (TDesc*)(base + ws_bytes);
    // the workspace header starts at zero (the kernels clear the rest they
    // read); the descriptor table goes up through kernel arguments
    hipLaunchKernelGGL(zero_words, dim3(1), dim3(64), 0, s, ws, 64);
    const uint32_t* src = (const uint32_t*)p.d.data();
    const size_t words = (size_t)T * sizeof(TDesc) / 4u;
    for (size_t at = 0; at < words; at += kBlobWords) {
        Blob b;
        const int cnt = (int)(words - at < (size_t)kBlobWords ? words - at : (size_t)kBlobWords);
        std::memcpy(b.w, src + at, (size_t)cnt * 4u);
        hipLaunchKernelGGL(put_words, dim3(1), dim3(256), 0, s, (uint32_t*)dd + at, b, cnt);
    }
    if (p.C > 0) {
        const uint32_t blocks = (p.C + 255u) / 256u < 1024u ? (p.C + 255u) / 256u : 1024u;
        hipLaunchKernelGGL(build_chunk_map, dim3(blocks), dim3(256), 0, s, (const TDesc*)dd, T, p.C);
    }
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) e = compress_launch(kind, ratio, seed, p, dd, out, carve_workspace(ws, p.plan), s);
    return e == hipSuccess ? BC_OK : BC_E_HIP;
}
