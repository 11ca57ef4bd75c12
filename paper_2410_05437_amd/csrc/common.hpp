// Device-side helpers shared by the gfx950 kernels of the projected linear layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace espace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// float -> bfloat16 with round-to-nearest-even; gfx950 converts two values
// per instruction (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint32_t bf16_rne(float f) { return pack_bf16x2(f, 0.f) & 0xffffu; }

__device__ __forceinline__ float bf16_to_f32(uint32_t h) {
    return __uint_as_float(h << 16);
}

// Zero the bfloat16 lanes e >= nvalid of an 8-element chunk (0 <= nvalid <= 8).
__device__ __forceinline__ u32x4_t mask_chunk(u32x4_t v, int nvalid) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const int e0 = 2 * w;
        uint32_t keep = (e0 + 1 < nvalid) ? 0xffffffffu : (e0 < nvalid ? 0x0000ffffu : 0u);
        v[w] &= keep;
    }
    return v;
}

// Load one 16-byte chunk of 8 bfloat16 values starting at element k of a row,
// keeping only elements k .. depth-1.  Chunks starting at or beyond `depth`
// are not read.  The row is padded to a multiple of 8 elements, so a partial
// chunk stays inside the row.
__device__ __forceinline__ u32x4_t load_chunk_masked(const uint16_t* row, int k, int depth) {
    u32x4_t v = {0u, 0u, 0u, 0u};
    const int nvalid = depth - k;
    if (nvalid > 0) {
        v = *reinterpret_cast<const u32x4_t*>(row + k);
        if (nvalid < 8) v = mask_chunk(v, nvalid);
    }
    return v;
}

// Branch-free variant for loops that keep many loads in flight: the chunk at
// element k of a row padded to a multiple of 8 elements, keeping `valid`
// elements (valid >= 8: all, valid <= 0: none; the address is then clamped
// to the row start so that the load stays inside the row).
__device__ __forceinline__ u32x4_t load_chunk_clamped(const uint16_t* row, int k, int valid) {
    const u32x4_t v = *reinterpret_cast<const u32x4_t*>(row + (valid > 0 ? k : 0));
    return mask_chunk(v, valid);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) {
    return __builtin_bit_cast(bf16x8_t, v);
}

// Bounded cross-workgroup waits (pair combine, readiness of the projection in
// the one-launch layer): a wait gives up after `spins` polls; the workgroup
// then writes NaN to the output it could not complete, so the failure is
// visible in the result, and counts the event in *timeouts, a device counter
// the host reads with espace_wait_timeouts().
__device__ __forceinline__ void note_timeout(const WaitCfg& w) {
    if (w.timeouts) atomicAdd(w.timeouts, 1ull);
}

// Workgroups are dispatched to the 8 XCDs of the chip round-robin by linear
// workgroup id.  Remap so that each XCD receives a contiguous range of tile
// indices (tiles next to each other share operand panels in that XCD's L2).
__device__ __forceinline__ int xcd_contiguous(int bid, int nblocks) {
    constexpr int NXCD = 8;
    const int q = nblocks / NXCD;
    const int r = nblocks % NXCD;
    const int x = bid % NXCD;
    const int i = bid / NXCD;
    return x * q + (x < r ? x : r) + i;
}

// Output-tile coordinates of workgroup bid among tiles_r x tiles_c tiles.
// map bit 0: skip the XCD remapping; bit 1: plain row-major order instead of
// groups of GROUP tile-rows walked column by column; bit 3: only the tiles on
// and above the diagonal of a square tiling (nblocks = n(n+1)/2 for
// tiles_c = n), row by row.
template <int GROUP>
__device__ __forceinline__ void tile_coords(int bid, int nblocks, int tiles_c, int map,
                                            int& tile_r, int& tile_c) {
    const int t = (map & 1) ? bid : xcd_contiguous(bid, nblocks);
    if (map & 8) {
        int r = 0, off = 0;
        while (r < tiles_c - 1 && off + (tiles_c - r) <= t) {
            off += tiles_c - r;
            ++r;
        }
        tile_r = r;
        tile_c = r + (t - off);
        return;
    }
    if (map & 2) {
        tile_r = t / tiles_c;
        tile_c = t - tile_r * tiles_c;
        return;
    }
    const int tiles_r = nblocks / tiles_c;
    const int group_size = GROUP * tiles_c;
    const int g = t / group_size;
    const int first_r = g * GROUP;
    const int gsz = (tiles_r - first_r) < GROUP ? (tiles_r - first_r) : GROUP;
    const int in_g = t - g * group_size;
    tile_r = first_r + in_g % gsz;
    tile_c = in_g / gsz;
}

}  // namespace espace
