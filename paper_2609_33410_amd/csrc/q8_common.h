// Pieces shared by the scans over a two-plane INT8 key cache: the integer
// matrix-core product, 2-byte scale loads, and where a 16-key chunk lives.
#pragma once

#include "decode_common.h"

namespace fold {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// C += A . B on a 16x16 tile with K = 64 INT8 (v_mfma_i32_16x16x64_i8); lane l
// holds 16 bytes of row l%16 of A and of column l%16 of B; C as the BF16 tiles.
__device__ __forceinline__ i32x4 mfma_i8(u32x4 a, u32x4 b, i32x4 c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, a),
                                               __builtin_bit_cast(i32x4, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t buf_load2(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, kStreamPolicy);
}

// Where a 16-key chunk lives: its first key row in the cache's element
// layout and its number of keys (0 past the sequence end or for a page id
// outside [0, num_pages)).  Buffer resources are built from it at each use,
// so a chunk in flight holds three scalar registers, not four resources.
struct Q8Loc {
  size_t row;
  uint32_t nk;
};

// Page of 16-key chunk c: pshift = log2(page_size / 16) when that is a power
// of two (a shift), else -1 (a division).
__device__ __forceinline__ int chunk_page_of(const ScanGeometry& g, int c, int pshift) {
  return pshift >= 0 ? c >> pshift : (c * kChunk) / g.page_size;
}

// Where chunk c lives, given its block-table entry phys (ignored for a
// contiguous view).
__device__ __forceinline__ Q8Loc q8_loc(const ScanGeometry& g, const ScanPlace& p, int c,
                                        int phys, int pshift) {
  Q8Loc l{0, 0};
  if (c < p.nchunks) {
    const int key0 = c * kChunk;
    bool ok = true;
    if (g.page_size > 0) {
      const int page = chunk_page_of(g, c, pshift);
      ok = phys >= 0 && phys < g.num_pages;
      l.row = (static_cast<size_t>(ok ? phys : 0) * g.hkv + p.kvh) * g.page_size +
              (key0 - page * g.page_size);
    } else {
      l.row = (static_cast<size_t>(p.seq) * g.hkv + p.kvh) * g.max_seq_len + key0;
    }
    if (ok) l.nk = static_cast<uint32_t>(min(kChunk, p.n - key0));
  }
  return l;
}

// Block-table entry of 16-key chunk c (0 for a contiguous view or past the
// sequence end); a scalar load.
__device__ __forceinline__ int q8_chunk_phys(const ScanGeometry& g, const ScanPlace& p, int c,
                                             int pshift) {
  if (g.page_size <= 0 || c >= p.nchunks) return 0;
  return ld_uniform(g.block_table,
                    static_cast<size_t>(p.seq) * g.max_pages + chunk_page_of(g, c, pshift));
}

// log2(page_size / 16) when that is a power of two, else -1 (see chunk_page_of).
__device__ __forceinline__ int q8_page_shift(const ScanGeometry& g) {
  if (g.page_size <= 0) return -1;
  const int cpp = g.page_size / kChunk;
  return (cpp & (cpp - 1)) == 0 ? __builtin_ctz(static_cast<unsigned>(cpp)) : -1;
}

}  // namespace fold
