// Pieces shared by the decode scan kernels: buffer resources over 16-key
// chunks, query-row lookup, and the chunk schedule of a split.
#pragma once

#include "fold_device.h"
#include "fold_internal.h"

namespace fold {

constexpr int kScanWaves = 4;
constexpr int kScanThreads = 64 * kScanWaves;
constexpr uint32_t kRsrcWord3 = 0x00020000u;  // raw buffer, 32-bit data (gfx9 family)
constexpr uint32_t kOutOfRange = 0x80000000u;  // an offset past any chunk resource

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// A buffer resource over `bytes` bytes at `base`: loads at offsets past the
// end return zero and touch no memory.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), static_cast<int>(kRsrcWord3));
}

// Cache policy of the cache-row stream: non-temporal (the NT bit of the gfx950
// cache-policy field).  A call reads each cached key and value row once; with
// this bit, randomly placed 4 KiB page slabs stream from HBM at about 6.6 TB/s
// against 5.9 TB/s with the default policy (measured on MI355X).
constexpr int kStreamPolicy = 2;

template <int POLICY = kStreamPolicy>
__device__ __forceinline__ u32x4 buf_load(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, POLICY);
}

struct RowInfo {
  int req;
  int head;
  bool ok;
};

// Query row rho of the rows attending (kv sequence seq, kv head kvh):
// rho = (position of the request in the sequence's row list) * G + (h mod G).
__device__ __forceinline__ RowInfo row_info(const ScanGeometry& g, int seq, int kvh, int rho,
                                            int nrows, int req0) {
  RowInfo ri;
  ri.ok = rho < nrows;
  const int rr = ri.ok ? rho : 0;
  ri.req = g.row_indptr ? ld_uniform(g.row_req, req0 + rr / g.group) : seq;
  ri.head = kvh * g.group + rr % g.group;
  ri.ok = ri.ok && ri.req >= 0 && ri.req < g.batch;
  return ri;
}

// Where one workgroup works: kv sequence, kv head, split, read group; the
// sequence's length and rows.  Block index order: sequence fastest, then kv
// head, split, read group.
struct ScanPlace {
  int seq, kvh, split, rg;
  int req0, nrows;
  int n, nchunks;
};

__device__ __forceinline__ ScanPlace scan_place(const DecodeArgs& a) {
  const ScanGeometry& g = a.geo;
  ScanPlace p;
  int bid = blockIdx.x;
  p.seq = bid % g.num_seqs;
  bid /= g.num_seqs;
  p.kvh = bid % g.hkv;
  bid /= g.hkv;
  p.split = bid % a.num_splits;
  p.rg = bid / a.num_splits;
  p.req0 = p.seq;
  int nreq = 1;
  if (g.row_indptr) {
    p.req0 = ld_uniform(g.row_indptr, p.seq);
    nreq = ld_uniform(g.row_indptr, p.seq + 1) - p.req0;
  }
  p.nrows = nreq * g.group;
  p.n = clamp_len(ld_uniform(g.seq_lens, p.seq), view_capacity(g));
  p.nchunks = (p.n + kChunk - 1) / kChunk;
  return p;
}

// Longest sequences first.  For a per-request view of at most kOrderMax
// sequences the block index runs over kv heads fastest, then splits, then the
// sequences by decreasing length (ties by index), then read groups.  Blocks
// are dispatched in index order as slots free up, so the workgroups of the
// longest sequences start first and the last to start are the shortest ones:
// a ragged batch drains with less of the call left to a half-empty chip.
// Which workgroup scans which keys changes nothing else (same sums, same
// bits).  Every thread of the workgroup must call it (one barrier).

__device__ __forceinline__ ScanPlace scan_place_by_length(const DecodeArgs& a, int* order) {
  const ScanGeometry& g = a.geo;
  const int cap = view_capacity(g);
  if (static_cast<int>(threadIdx.x) < g.num_seqs) {
    const int i = threadIdx.x;
    const int li = clamp_len(g.seq_lens[i], cap);
    int r = 0;
    for (int j = 0; j < g.num_seqs; ++j) {
      const int lj = clamp_len(g.seq_lens[j], cap);
      r += (lj > li || (lj == li && j < i)) ? 1 : 0;
    }
    order[r] = i;
  }
  __syncthreads();
  ScanPlace p;
  int bid = blockIdx.x;
  p.kvh = bid % g.hkv;
  bid /= g.hkv;
  p.split = bid % a.num_splits;
  bid /= a.num_splits;
  const int rank = bid % g.num_seqs;
  p.rg = bid / g.num_seqs;
  p.seq = __builtin_amdgcn_readfirstlane(order[rank]);
  p.req0 = p.seq;
  p.nrows = g.group;
  p.n = clamp_len(ld_uniform(g.seq_lens, p.seq), cap);
  p.nchunks = (p.n + kChunk - 1) / kChunk;
  return p;
}

// Block-table entry of the page holding 16-key chunk c of the sequence (0 for
// a contiguous view or past the sequence end).  A scalar load: issuing it well
// before chunk_rsrc_at() hides its latency.
__device__ __forceinline__ int chunk_page(const ScanGeometry& g, const ScanPlace& p, int c) {
  if (g.page_size <= 0 || c >= p.nchunks) return 0;
  return ld_uniform(g.block_table,
                    static_cast<size_t>(p.seq) * g.max_pages + (c * kChunk) / g.page_size);
}

// Buffer resources over the valid keys of 16-key chunk c of (seq, kvh), given
// the chunk's block-table entry: empty past the sequence end or for a page id
// outside [0, num_pages).
template <int D>
__device__ __forceinline__ void chunk_rsrc_at(const ScanGeometry& g, const ScanPlace& p, int c,
                                              int phys, rsrc_t* rk, rsrc_t* rv) {
  const uint16_t* kb = g.k;
  const uint16_t* vb = g.v;
  uint32_t bytes = 0;
  if (c < p.nchunks) {
    const int key0 = c * kChunk;
    const int nk = min(kChunk, p.n - key0);
    size_t off;
    bool ok = true;
    if (g.page_size > 0) {
      const int page = key0 / g.page_size;
      ok = phys >= 0 && phys < g.num_pages;
      off = ((static_cast<size_t>(ok ? phys : 0) * g.hkv + p.kvh) * g.page_size +
             (key0 - page * g.page_size)) * D;
    } else {
      off = ((static_cast<size_t>(p.seq) * g.hkv + p.kvh) * g.max_seq_len + key0) * D;
    }
    if (ok) {
      kb += off;
      vb += off;
      bytes = static_cast<uint32_t>(nk) * D * 2;
    }
  }
  *rk = make_rsrc(kb, bytes);
  *rv = make_rsrc(vb, bytes);
}

template <int D>
__device__ __forceinline__ void chunk_rsrc(const ScanGeometry& g, const ScanPlace& p, int c,
                                           rsrc_t* rk, rsrc_t* rv) {
  chunk_rsrc_at<D>(g, p, c, chunk_page(g, p, c), rk, rv);
}

}  // namespace fold
