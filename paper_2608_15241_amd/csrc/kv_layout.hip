// local_kv_pool_import / local_kv_pool_export: the paged KV pool between the
// token-major layout [num_blocks][Hkv][16][D] (a block's 16 slots in order,
// each slot's D values contiguous: the layout a serving stack commonly keeps,
// §2.2 "KV cache") and this library's K [num_blocks][Hkv][D/8][16][8] and
// V [num_blocks][Hkv][D][16] layouts.
//
// Design (HBM-bound: every byte read once, written once): a workgroup of 256
// threads per (block, head) tile pair, a grid-stride loop over the tiles.
// K moves as 16-byte pieces (8 dims of one slot are contiguous in both
// layouts; only the pieces' order changes), so a thread copies its pieces
// register to register, the writes of consecutive threads contiguous. V is a
// 2-byte transpose (slot-major <-> dim-major) through LDS: 16-byte reads,
// 2-byte LDS traffic, 16-byte writes.
#include "common.hpp"

namespace localk {
namespace {

constexpr int kLayThreads = 256;

// token-major -> library (IMPORT) or library -> token-major (!IMPORT)
template <int D, bool IMPORT>
__global__ __launch_bounds__(kLayThreads) void kv_layout_kernel(
    const uint16_t* __restrict__ k_src, const uint16_t* __restrict__ v_src,
    uint16_t* __restrict__ k_dst, uint16_t* __restrict__ v_dst, int64_t tiles) {
  constexpr int C8 = D / 8;                    // 16-byte pieces per slot
  constexpr int PIECES = kBlockSize * C8;      // per tile (256 or 128)
  constexpr int TILE = kBlockSize * D;         // elements per tile
  __shared__ uint16_t vt[D][kBlockSize + 2];   // V of the tile, dim-major (+2: banks)
  const int tid = threadIdx.x;
  for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    const int64_t base = tile * TILE;
    if (tid < PIECES) {
      // K piece (slot, dims 8c .. 8c+7); thread t takes library position t,
      // i.e. c = t / 16, slot = t % 16
      const int c = tid / kBlockSize, slot = tid % kBlockSize;
      const int64_t lib_off = base + (static_cast<int64_t>(c) * kBlockSize + slot) * 8;
      const int64_t tok_off = base + static_cast<int64_t>(slot) * D + 8 * c;
      const u32x4 kv = ld_global<u32x4>(k_src + (IMPORT ? tok_off : lib_off));
      *reinterpret_cast<u32x4*>(k_dst + (IMPORT ? lib_off : tok_off)) = kv;
    }
    if (IMPORT) {
      // V: slot-major pieces into LDS, dim rows of 16 slots out
      if (tid < PIECES) {
        const int slot = tid / C8, c = tid % C8;
        const u32x4 vv = ld_global<u32x4>(v_src + base + static_cast<int64_t>(slot) * D + 8 * c);
        const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          vt[8 * c + 2 * q][slot] = static_cast<uint16_t>(w[q] & 0xffffu);
          vt[8 * c + 2 * q + 1][slot] = static_cast<uint16_t>(w[q] >> 16);
        }
      }
      __syncthreads();
      for (int e = tid; e < 2 * D; e += kLayThreads) {
        const int d = e / 2, h = e % 2;
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          w[q] = static_cast<uint32_t>(vt[d][8 * h + 2 * q]) |
                 (static_cast<uint32_t>(vt[d][8 * h + 2 * q + 1]) << 16);
        *reinterpret_cast<u32x4*>(v_dst + base + d * kBlockSize + 8 * h) =
            u32x4{w[0], w[1], w[2], w[3]};
      }
    } else {
      // V: dim rows (two 16-byte halves each) into LDS, slot-major pieces out
      for (int e = tid; e < 2 * D; e += kLayThreads) {
        const int d = e / 2, h = e % 2;
        const u32x4 vv = ld_global<u32x4>(v_src + base + d * kBlockSize + 8 * h);
        const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          vt[d][8 * h + 2 * q] = static_cast<uint16_t>(w[q] & 0xffffu);
          vt[d][8 * h + 2 * q + 1] = static_cast<uint16_t>(w[q] >> 16);
        }
      }
      __syncthreads();
      if (tid < PIECES) {
        const int slot = tid / C8, c = tid % C8;
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          w[q] = static_cast<uint32_t>(vt[8 * c + 2 * q][slot]) |
                 (static_cast<uint32_t>(vt[8 * c + 2 * q + 1][slot]) << 16);
        *reinterpret_cast<u32x4*>(v_dst + base + static_cast<int64_t>(slot) * D + 8 * c) =
            u32x4{w[0], w[1], w[2], w[3]};
      }
    }
    __syncthreads();  // before the next tile rewrites vt
  }
}

template <bool IMPORT>
local_status_t kv_layout(const uint16_t* k_src, const uint16_t* v_src, int64_t num_blocks,
                         int32_t Hkv, int32_t D, int32_t block_size, uint16_t* k_dst,
                         uint16_t* v_dst, void* stream, const char* who) {
  if (num_blocks < 0 || Hkv < 1)
    return local_fail(LOCAL_ERR_SHAPE, "%s: num_blocks %lld, Hkv %d", who,
                      (long long)num_blocks, Hkv);
  if (D != 64 && D != 128)
    return local_fail(LOCAL_ERR_UNSUPPORTED, "%s: D must be 64 or 128, got %d", who, D);
  if (block_size != kBlockSize)
    return local_fail(LOCAL_ERR_UNSUPPORTED, "%s: block_size must be 16, got %d", who,
                      block_size);
  if (num_blocks == 0) return LOCAL_OK;  // nothing to read or write
  if (!k_src || !v_src || !k_dst || !v_dst)
    return local_fail(LOCAL_ERR_NULL, "%s: NULL pool pointer", who);
  const int64_t tiles = num_blocks * Hkv;
  const int64_t bytes = tiles * kBlockSize * D * 2;
  auto overlap = [&](const void* a, const void* b) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + static_cast<uintptr_t>(bytes) && y < x + static_cast<uintptr_t>(bytes);
  };
  if (overlap(k_src, k_dst) || overlap(k_src, v_dst) || overlap(v_src, k_dst) ||
      overlap(v_src, v_dst) || overlap(k_dst, v_dst))
    return local_fail(LOCAL_ERR_SHAPE, "%s: the pools overlap (the conversion is not in place)",
                      who);
  const unsigned grid = static_cast<unsigned>(tiles < 65536 ? tiles : 65536);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (D == 64)
    kv_layout_kernel<64, IMPORT><<<grid, kLayThreads, 0, s>>>(k_src, v_src, k_dst, v_dst, tiles);
  else
    kv_layout_kernel<128, IMPORT><<<grid, kLayThreads, 0, s>>>(k_src, v_src, k_dst, v_dst, tiles);
  return local_check_launch(who);
}

}  // namespace
}  // namespace localk

extern "C" local_status_t local_kv_pool_import(const uint16_t* k_tok, const uint16_t* v_tok,
                                               int64_t num_blocks, int32_t Hkv, int32_t D,
                                               int32_t block_size, uint16_t* k_cache,
                                               uint16_t* v_cache, void* stream) {
  return localk::kv_layout<true>(k_tok, v_tok, num_blocks, Hkv, D, block_size, k_cache, v_cache,
                                 stream, "kv_pool_import");
}

extern "C" local_status_t local_kv_pool_export(const uint16_t* k_cache, const uint16_t* v_cache,
                                               int64_t num_blocks, int32_t Hkv, int32_t D,
                                               int32_t block_size, uint16_t* k_tok,
                                               uint16_t* v_tok, void* stream) {
  return localk::kv_layout<false>(k_cache, v_cache, num_blocks, Hkv, D, block_size, k_tok, v_tok,
                                  stream, "kv_pool_export");
}
