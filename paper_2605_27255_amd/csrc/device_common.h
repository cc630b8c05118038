// Device helpers shared by the gfx950 kernels: bf16 storage, the 16x16x32
// bf16 MFMA, wave reductions, the tiled operand layout and SplitMix64.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pipo {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kWave = 64;

// ---- bf16 storage (uint16 bit patterns) ----------------------------------
__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
// Round to nearest even; inputs here are finite.
__device__ __forceinline__ uint32_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
    return f2bf(lo) | (f2bf(hi) << 16);
}
// Two floats into one bf16x2 word (element lo in the low half), rounded to
// nearest even by the hardware conversion (v_cvt_pk_bf16_f32); for finite
// inputs the same bits as f2bf.
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
__device__ __forceinline__ uint32_t pack_bf2_hw(float lo, float hi) {
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
// x ~= bf(hi) + bf(lo): the bf16 rounding of x and of its remainder.
__device__ __forceinline__ void split_bf(float x, uint32_t &hi, uint32_t &lo) {
    hi = f2bf(x);
    lo = f2bf(x - bf2f(hi));
}
// Eight floats into hi and lo bf16x8 words.
__device__ __forceinline__ void split8(const float *v, u32x4 &hi, u32x4 &lo) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t h = pack_bf2_hw(v[2 * i], v[2 * i + 1]);
        hi[i] = h;
        lo[i] = pack_bf2_hw(v[2 * i] - bf_lo(h), v[2 * i + 1] - bf_hi(h));
    }
}

// ---- MFMA: C[16x16] += A[16x32] * B[32x16], bf16 in, fp32 accumulate ------
// Lane l = 16*g + r supplies A row r and B column r, eight k-elements each
// (group g); element e of A's lane (r, g) multiplies element e of B's lane
// (c, g).  Accumulator lane l holds C[4*(l/16) + v][l % 16], v = 0..3.
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// ---- wave reductions -------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
// The same sum without LDS traffic: DPP within each 16-lane row (pairs,
// quads, half-row and row mirrors), then the four row sums read into scalar
// registers and added in row order; every lane gets the result.
#define PIPO_DPP(v, ctrl) \
    __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, (v)), (ctrl), 0xF, 0xF, false))
__device__ __forceinline__ float wave_sum_dpp(float v) {
    v += PIPO_DPP(v, 0xB1);    // quad_perm [1,0,3,2]
    v += PIPO_DPP(v, 0x4E);    // quad_perm [2,3,0,1]
    v += PIPO_DPP(v, 0x141);   // row_half_mirror
    v += PIPO_DPP(v, 0x140);   // row_mirror
    const int u = __builtin_bit_cast(int, v);
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(u, 0)) +
           __builtin_bit_cast(float, __builtin_amdgcn_readlane(u, 16)) +
           __builtin_bit_cast(float, __builtin_amdgcn_readlane(u, 32)) +
           __builtin_bit_cast(float, __builtin_amdgcn_readlane(u, 48));
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
// Sum over the four lanes that share l % 16 (the accumulator column).
__device__ __forceinline__ float col_sum(float v) {
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
}
__device__ __forceinline__ float col_max(float v) {
    v = fmaxf(v, __shfl_xor(v, 16));
    v = fmaxf(v, __shfl_xor(v, 32));
    return v;
}

// ---- tiled operand layout ---------------------------------------------------
// A matrix [R][K] (R % 16 == 0, K % 32 == 0) is stored as 16x32 tiles of 1 KB,
// tile (R/16 row-strip, k/32) at ((r/16)*(K/32) + k/32)*512 elements; inside a
// tile the 16 bytes of lane l = 16*(k%32/8) + r%16 hold k%8 = 0..7, so a
// wave's 16-byte-per-lane load of a tile is one contiguous 1 KB read and is
// directly an MFMA A or B operand.
__host__ __device__ __forceinline__ int64_t tiled_index(int64_t r, int64_t k, int64_t K) {
    return (((r >> 4) * (K >> 5) + (k >> 5)) << 9) + ((((k & 31) >> 3) * 16 + (r & 15)) << 3) + (k & 7);
}

// ---- V cache tile order ------------------------------------------------------
// Slot of key kappa (0..31) inside a 32-key V tile [d][32]: the order in which
// the attention kernels hold probabilities as MFMA B operands (accumulator
// lane group g, element v of 16-key tile tau holds key 16 tau + 4 g + v).
__host__ __device__ __forceinline__ int vslot(int kappa) {
    return 8 * ((kappa & 15) >> 2) + 4 * (kappa >> 4) + (kappa & 3);
}

// ---- SplitMix64 (Steele, Lea and Flood, OOPSLA 2014), as a stateless hash --
__host__ __device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
__host__ __device__ __forceinline__ uint64_t rng_key(uint64_t seed, uint64_t tid) {
    return splitmix64(seed ^ splitmix64(tid));
}

// ---- argmax keys ------------------------------------------------------------
// A 64-bit key whose unsigned maximum is the largest value and, among equal
// values, the lowest id: order-preserving float bits above the inverted id.
__device__ __forceinline__ uint64_t argmax_key(float v, uint32_t id) {
    uint32_t u = __float_as_uint(v);
    u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((uint64_t)u << 32) | (uint64_t)(0xFFFFFFFFu - id);
}
__device__ __forceinline__ int32_t argmax_key_id(uint64_t key) {
    return (int32_t)(0xFFFFFFFFu - (uint32_t)(key & 0xFFFFFFFFull));
}
// A token id used as a row index, forced into [0, vocab).
__device__ __forceinline__ int clamp_id(int id, int vocab) {
    return id < 0 ? 0 : (id >= vocab ? vocab - 1 : id);
}

}  // namespace pipo
