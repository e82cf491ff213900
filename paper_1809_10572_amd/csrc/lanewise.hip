// Lane-wise SAMD arithmetic on packed words (Sec. 3, conventional SAMD arithmetic, and
// Sec. 4, vector scale): every uint32 word of the packed format holds P = 32 / b lanes
// of b bits, lane i in bits [i b, i b + b), the bits above lane P - 1 zero.  Each
// operation works on whole words with scalar integer instructions; the spacer is
// temporary (the top bit of every lane), so the words keep the dense storage format.
// Results are the lane values modulo 2^b: two's-complement wrap-around for signed
// formats, the same bit patterns.
#include <hip/hip_runtime.h>

#include "hip_util.hpp"

namespace samd {

namespace {

// Per-format lane masks of one 32-bit word: the valid lanes, their top bits, their
// bottom bits, the even and the odd lanes.
template <int B>
struct LaneMasks {
    static constexpr int P = 32 / B;
    static constexpr uint32_t valid = P * B == 32 ? 0xffffffffu : (1u << (P * B)) - 1;
    static constexpr uint32_t lsb() {
        uint32_t m = 0;
        for (int i = 0; i < P; ++i) m |= 1u << (i * B);
        return m;
    }
    static constexpr uint32_t msb = lsb() << (B - 1);
    static constexpr uint32_t even() {
        uint32_t m = 0;
        for (int i = 0; i < P; i += 2) m |= ((1u << B) - 1) << (i * B);
        return m;
    }
    static constexpr uint32_t odd = valid & ~even();
};

// Lane-wise add with a temporary spacer (each lane's top bit): the low bits are added
// with one scalar add (a carry stops in the top bit), and the top bit is rebuilt as the
// xor of both top bits and that carry.
template <int B>
__device__ __forceinline__ uint32_t lane_add(uint32_t a, uint32_t b) {
    using Mk = LaneMasks<B>;
    constexpr uint32_t low = Mk::valid & ~Mk::msb;
    return (((a & low) + (b & low)) ^ ((a ^ b) & Mk::msb)) & Mk::valid;
}

// Lane-wise subtract: every minuend top bit is forced to 1 so no borrow leaves its lane,
// then the top bit is corrected.
template <int B>
__device__ __forceinline__ uint32_t lane_sub(uint32_t a, uint32_t b) {
    using Mk = LaneMasks<B>;
    constexpr uint32_t low = Mk::valid & ~Mk::msb;
    const uint32_t diff = (a | Mk::msb) - (b & low);
    return (diff ^ ((a ^ b) & Mk::msb) ^ Mk::msb) & Mk::valid;
}

// Lane-wise product modulo 2^b by shift and add, b steps (lane-wise multiply figure):
// step k adds a * 2^k into the lanes whose multiplier has bit k set, masked to the
// lane's bits k .. b-1 (bits shifted in from the lane below are excluded).
template <int B>
__device__ __forceinline__ uint32_t lane_mul(uint32_t a, uint32_t b) {
    using Mk = LaneMasks<B>;
    uint32_t acc = 0, probe = Mk::lsb();
#pragma unroll
    for (int k = 0; k < B; ++k) {
        const uint32_t sel = b & probe;
        const uint32_t fill = (sel << (B - k)) - sel;   // bits k .. b-1 of the selected lanes
        acc = lane_add<B>(acc, a & fill);
        a <<= 1;
        probe <<= 1;
    }
    return acc;
}

// Vector scale modulo 2^b (scale-wrap figure): the even and the odd lanes each get b
// zero bits above them, so one multiply by the b-bit scalar leaves every 2b-bit product
// in its lane and the cleared lane above; each lane keeps its low b bits.
template <int B>
__device__ __forceinline__ uint32_t lane_scale(uint32_t a, uint32_t s) {
    using Mk = LaneMasks<B>;
    return (((a & Mk::even()) * s) & Mk::even()) | (((a & Mk::odd) * s) & Mk::odd);
}

// One thread per 16 bytes (four words), grid-stride; the tail word by word.
template <int B, int OP>
__global__ __launch_bounds__(256) void lanewise_kernel(const uint32_t *__restrict__ a, const uint32_t *__restrict__ b,
                                                       int64_t nwords, uint32_t scalar, uint32_t *__restrict__ dst) {
    auto op = [&](uint32_t x, uint32_t y) -> uint32_t {
        if constexpr (OP == SAMD_LANE_ADD) return lane_add<B>(x, y);
        else if constexpr (OP == SAMD_LANE_SUB) return lane_sub<B>(x, y);
        else if constexpr (OP == SAMD_LANE_MUL) return lane_mul<B>(x, y);
        else return lane_scale<B>(x, scalar);
    };
    const int64_t nvec = nwords / 4;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nvec; i += stride) {
        const uint4 x = ((const uint4 *)a)[i];
        const uint4 y = OP == SAMD_LANE_SCALE ? x : ((const uint4 *)b)[i];
        ((uint4 *)dst)[i] = uint4{op(x.x, y.x), op(x.y, y.y), op(x.z, y.z), op(x.w, y.w)};
    }
    for (int64_t w = nvec * 4 + (int64_t)blockIdx.x * 256 + threadIdx.x; w < nwords; w += stride)
        dst[w] = op(a[w], OP == SAMD_LANE_SCALE ? 0u : b[w]);
}

}  // namespace

int launch_lanewise(int op, const uint32_t *a, const uint32_t *b, int64_t nwords, int bits, uint32_t scalar,
                    uint32_t *dst, hipStream_t s) {
    const int grid = grid_for((nwords + 3) / 4, 256);
    bool launched = false;
#define SAMD_LANE_CASE(B_, OP_)                                                                          \
    if (!launched && bits == B_ && op == OP_) {                                                          \
        hipLaunchKernelGGL((lanewise_kernel<B_, OP_>), dim3(grid), dim3(256), 0, s, a, b, nwords, scalar, dst); \
        launched = true;                                                                                 \
    }
#define SAMD_LANE_OPS(B_) \
    SAMD_LANE_CASE(B_, SAMD_LANE_ADD) SAMD_LANE_CASE(B_, SAMD_LANE_SUB) SAMD_LANE_CASE(B_, SAMD_LANE_MUL) \
    SAMD_LANE_CASE(B_, SAMD_LANE_SCALE)
    SAMD_LANE_OPS(1) SAMD_LANE_OPS(2) SAMD_LANE_OPS(3) SAMD_LANE_OPS(4)
    SAMD_LANE_OPS(5) SAMD_LANE_OPS(6) SAMD_LANE_OPS(7) SAMD_LANE_OPS(8)
#undef SAMD_LANE_OPS
#undef SAMD_LANE_CASE
    if (!launched) {
        set_error("lane-wise: no kernel for this operation");
        return SAMD_EINVAL;
    }
    return check_launch("lane-wise arithmetic");
}

}  // namespace samd
