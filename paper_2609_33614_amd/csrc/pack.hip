// Packed expert-weight layout (gfx950).
//
// A row-major weight matrix W [groups][M][K] (bf16) is stored as blocks of
// 16 rows x 32 reduction elements, 1 KB each, in the order
//   block (g, rb, ks) at index (g * M / 16 + rb) * K / 32 + ks,
// and inside a block in the lane order of the MFMA A operand: the 16-byte
// fragment of lane l = 16 q + i holds W[g][16 rb + i][32 ks + 8 q .. + 7].
// A wave that owns 16 weight rows then reads each k-step of them as one
// contiguous kilobyte, which the decode kernels load with the streaming
// cache policy; the prefill tiles gather the same fragments into their LDS
// rows.  Packing is a permutation: results are bit-identical to the
// row-major layout.
#include "eat_device.h"
#include "eat_internal.h"

namespace eat {
namespace {

constexpr int kThreads = 256;

// one thread per 16-byte fragment, in destination order (writes coalesce)
__global__ __launch_bounds__(kThreads) void pack_kernel(const uint16_t* __restrict__ src, int64_t frags, int M,
                                                        int K, uint16_t* __restrict__ dst) {
    const int kb = K / 32;
    for (int64_t f = blockIdx.x * int64_t(kThreads) + threadIdx.x; f < frags; f += int64_t(gridDim.x) * kThreads) {
        const int lane = static_cast<int>(f & 63);
        const int64_t blk = f >> 6;
        const int ks = static_cast<int>(blk % kb);
        const int64_t grb = blk / kb;                       // g * M / 16 + rb
        const int64_t row = grb * 16 + (lane & 15);         // row of the [groups * M][K] matrix
        const int col = 32 * ks + 8 * (lane >> 4);
        *reinterpret_cast<bf16x8*>(dst + 8 * f) = *reinterpret_cast<const bf16x8*>(src + row * K + col);
    }
}

}  // namespace

hipError_t launch_pack(const uint16_t* src, int32_t groups, int32_t M, int32_t K, uint16_t* dst, hipStream_t s) {
    const int64_t frags = static_cast<int64_t>(groups) * M * K / 8;
    if (frags == 0) return hipSuccess;
    const int grid = static_cast<int>(std::min<int64_t>((frags + kThreads - 1) / kThreads, 16384));
    pack_kernel<<<grid, kThreads, 0, s>>>(src, frags, M, K, dst);
    return hipGetLastError();
}

}  // namespace eat
