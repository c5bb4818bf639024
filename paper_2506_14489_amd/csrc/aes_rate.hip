// The AES of the projection-gate hash alone, for measuring the device's AES
// rate: AES-128 under the hash key in counter mode, in two formulations.
//
//  * k_aes_ctr: the evaluator's round code (two replicated round tables in
//    LDS, one v_perm_b32 per lookup address; device.hpp), four blocks per
//    lane interleaved as in a two-gate evaluator step.
//  * k_aes_ctr_bs: bitsliced, 32 blocks per lane (aes_bitslice.hpp): no
//    table lookups, every operation on the vector ALU, with the transposes
//    into and out of bit slices.
//
// Both write d_out[4i .. 4i+3] = AES_K(c0 + i) (see include/redash.h).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/redash.h"
#include "aes_bitslice.hpp"
#include "device.hpp"

namespace redash {

namespace {

constexpr int kCtrBlock = 768;  // as the evaluator: two workgroups of 12 waves per CU
constexpr int kCtrWaves = 6;
constexpr uint32_t kCtrLds = kTableRegionBytes + 4 * kLdsKeyWords;  // round tables, then the key

}  // namespace

template <int BLOCK>
__global__ void __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(kCtrWaves, kCtrWaves)))
k_aes_ctr(uint64_t count, uint64_t c0, uint32_t *__restrict__ out) {
    extern __shared__ uint32_t lds[];
    uint32_t *K = lds + kTableRegionBytes / 4;
    stage_perm_te02(lds, threadIdx.x, blockDim.x);
    stage_hash_key(K, threadIdx.x, blockDim.x);
    __syncthreads();
    const PermTE02 TT = perm_te02();
    const uint64_t nthr = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    const uint64_t groups = (count + 3) / 4;
    for (uint64_t t = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < groups; t += nthr) {
        uint32_t s[4][4];
        static_for<4>([&](auto b) {
            const uint64_t c = c0 + 4 * t + b;  // the counter block, mod 2^128 (c0 < 2^64)
            s[b][0] = static_cast<uint32_t>(c);
            s[b][1] = static_cast<uint32_t>(c >> 32);
            s[b][2] = (c < c0) ? 1u : 0u;
            s[b][3] = 0;
        });
        aes128_encrypt_n<4>(TT, s, LdsKey{K});
        static_for<4>([&](auto b) {
            if (4 * t + b < count) {
                uint4 v;
                v.x = s[b][0];
                v.y = s[b][1];
                v.z = s[b][2];
                v.w = s[b][3];
                *reinterpret_cast<uint4 *>(out + 4 * (4 * t + b)) = v;
            }
        });
    }
}

// Thread t takes blocks 32t' .. 32t'+31 for t' = t, t + T, ...: the counter
// words of its 32 blocks are transposed into bit slices (three 32 x 32 bit
// transposes; the top word is 0), encrypted, and transposed back.
//
// The 128 state slices and the S-box temporaries need about 256 VGPRs: two
// waves per SIMD (1.4x the rate of one wave per SIMD at 272 registers; at
// three waves the allocator spills 484 bytes per lane).
template <int BLOCK>
__global__ void __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_aes_ctr_bs(uint64_t count, uint64_t c0, uint32_t *__restrict__ out) {
    const uint64_t nthr = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    const uint64_t groups = (count + 31) / 32;
    for (uint64_t t = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < groups; t += nthr) {
        uint32_t st[16][8];
        static_for<4>([&](auto w) {
            uint32_t a[32];
            static_for<32>([&](auto i) {
                const uint64_t c = c0 + 32 * t + i;
                a[i] = w == 0 ? static_cast<uint32_t>(c) : w == 1 ? static_cast<uint32_t>(c >> 32)
                                                         : w == 2 ? ((c < c0) ? 1u : 0u) : 0u;
            });
            if (w < 3) transpose32(a);
            static_for<32>([&](auto q) { st[4 * w + q / 8][q % 8] = a[q]; });
        });
        aes128_bs(st);
        static_for<4>([&](auto w) {
            uint32_t a[32];
            static_for<32>([&](auto q) { a[q] = st[4 * w + q / 8][q % 8]; });
            transpose32(a);
            static_for<32>([&](auto i) {
                if (32 * t + i < count) out[4 * (32 * t + i) + w] = a[i];
            });
        });
    }
}

}  // namespace redash

using namespace redash;

namespace {

int launched() { return hipGetLastError() == hipSuccess ? REDASH_OK : REDASH_E_HIP; }

int compute_units(uint64_t *out) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return REDASH_E_HIP;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        return REDASH_E_HIP;
    *out = static_cast<uint64_t>(cus);
    return REDASH_OK;
}

}  // namespace

extern "C" {

int redash_aes_ctr(uint64_t count, uint64_t c0, uint32_t *d_out, hipStream_t stream) {
    if (count == 0) return REDASH_OK;
    if (!d_out) return REDASH_E_NULL;
    if (count > (1ull << 40)) return REDASH_E_PARAM;
    uint64_t cus = 0;
    int rc = compute_units(&cus);
    if (rc) return rc;
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(&k_aes_ctr<kCtrBlock>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kCtrLds)) != hipSuccess)
        return REDASH_E_HIP;
    // at most one round of two workgroups per CU; each thread loops over its groups of four
    const uint64_t groups = (count + 3) / 4;
    const uint64_t grid = std::min<uint64_t>(2 * cus, (groups + kCtrBlock - 1) / kCtrBlock);
    hipLaunchKernelGGL(k_aes_ctr<kCtrBlock>, dim3(static_cast<unsigned>(grid)), dim3(kCtrBlock), kCtrLds, stream,
                       count, c0, d_out);
    return launched();
}

int redash_aes_ctr_bitsliced(uint64_t count, uint64_t c0, uint32_t *d_out, hipStream_t stream) {
    if (count == 0) return REDASH_OK;
    if (!d_out) return REDASH_E_NULL;
    if (count > (1ull << 40)) return REDASH_E_PARAM;
    uint64_t cus = 0;
    int rc = compute_units(&cus);
    if (rc) return rc;
    constexpr int block = 256;
    // four rounds of two workgroups per CU (measured 6% faster than one round)
    const uint64_t groups = (count + 31) / 32;
    const uint64_t grid = std::min<uint64_t>(8 * cus, (groups + block - 1) / block);
    hipLaunchKernelGGL(k_aes_ctr_bs<block>, dim3(static_cast<unsigned>(grid)), dim3(block), 0, stream, count, c0,
                       d_out);
    return launched();
}

}  // extern "C"
