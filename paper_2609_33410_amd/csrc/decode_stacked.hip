// Decode scan for stacked query rows: a kv sequence attended by more than 32
// query rows, as at the prefix level of a shared-prefix cascade (Section 4
// "Value product": a shared prefix is decoded once with the rows of all its
// requests stacked; Appendix E: past 64 rows the level runs on a kernel laid
// out as prefill is; Algorithm 1).
//
// Workgroup = (kv sequence, kv head, split, read group of 64 rows); eight
// wave64s.  Wave w owns the 16-row block w%4 of the read group and the key half
// w/4 (keys 32(w/4) .. +32) of every 64-key tile of the split.  Each K and V
// tile therefore leaves memory once per 64 rows and is shared through LDS:
//
//   fetch    every wave DMAs its eighth of the tile (keys 8w .. 8w+8) from
//            memory into LDS (buffer_load_dwordx4 ... lds, no registers).  The
//            16-byte chunks of a key row are permuted (slot = chunk ^ f(key)) so
//            that the operand reads below touch each of the 64 LDS banks once
//            per 256 bytes.
//   scores   S^T[key][row] = K . Q^T with v_mfma_f32_16x16x32_bf16 for two
//            16-key subtiles: keys on M (read from LDS), the wave's rows on N
//            (Q^T in registers), channels on K.  Lane l holds keys 4(l/16)+i of
//            row l%16 in each subtile.
//   verdict  x = s - Z_i (FP32 FMA); live = x >= -T; the live bits of the 64
//            rows are ORed (DPP within a wave, LDS across waves) into the tile's
//            64-bit read mask, and only live value rows are fetched (the others
//            get an offset past the chunk's buffer resource: zeros land in LDS,
//            no bytes move).
//   product  A^T[d][row] += V^T[d][key] . P^T[key][row] with
//            v_mfma_f32_16x16x32_bf16 over the wave's 32 keys.  The reduction
//            slots 8(l/16) .. +8 of lane l hold keys 4(l/16)+i of the two
//            subtiles, so P^T is the score output's own register layout, and
//            the matching V^T operand is two transposing LDS reads
//            (ds_read_b64_tr_b16).  The weight enters as bf16(hi) +
//            bf16(residual), two products; L adds the FP32 weight of every key.
//
// F16 (the stacked level of a two-plane key cache; Appendix E, tile layouts):
// the K tiles hold FP16 keys fp16(e (a + b/256)) written once per prefix, the
// query operand is fp16(qa + qb/256) formed from the query codes in the
// prologue, the scores run on v_mfma_f32_16x16x32_f16 and x = eta_i s - Z_i.
// Everything else is the BF16 kernel's.
//
// CX (block model of BF16 values, finite T): each weighed 16-key chunk's cut
// mass per row, the summed weights of its cut keys, is also written to
// chunk_cut.
//
// CASC (fold_decode_cascade): after the prefix tiles of its split, a
// workgroup scans the suffix tiles of its read group's requests that fall to
// the split, through the same pipeline, and adds them to the same slot (pairs
// add; Section 4, "Value product").  A suffix tile weighs only the rows of
// its own request.  LC: the finite-depth cut mass is accumulated only when
// the caller asked for it (part_Lcut).
//
// Pipelines.  Dense (T = inf): keys run one tile ahead of values; while the
// product of tile t runs on the matrix cores, the weights of tile t+1 are
// formed, and keys of t+4 / values of t+3 are in flight (four stages each).
// Gated: keys run two tiles ahead; tile t+2 is scored and its live value rows
// requested while the product of tile t runs (four key and three value
// stages).  EAGER (finite T, the production kernel): the dense pipeline with
// the depth rule deciding every weight, so value rows are fetched with their
// keys.  A stacked level reads a few MB per call and is bound by per-wave
// latency, not by HBM: waiting for a tile's verdict before its values move
// costs more than the bytes it saves (measured slower at every depth from 2
// to 16 on the 512 x 16384 cascade prefix, with as few as 0.8% of its pages
// live).  Cut keys' values meet a zero weight, so the slots hold the same
// bits as the gated fetch's, which the debug variant keeps (its read bits are
// the ones the tests check).  The DMAs are issued from assembly, so the compiler's wait
// insertion does not see them and never drains the prefetch; every wait for
// them is explicit (s_waitcnt vmcnt + an LDS-only barrier).  The two key halves
// of a row block add their partials in LDS at the end, in a fixed order.
#include <type_traits>

#include "decode_common.h"

namespace fold {
namespace {

constexpr int kStkWaves = 8;
constexpr int kStkThreads = 64 * kStkWaves;
constexpr int kStkRows = 64;  // rows per read group: four blocks of 16
constexpr int kWaveSize = 64;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Wait until at most N of this wave's vector-memory loads are outstanding
// (gfx9 s_waitcnt: vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt at their
// maxima, i.e. not waited for).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Wait until at most U * L loads are outstanding, U a wave-uniform count of
// load groups of L instructions each (0 <= U <= 7).
template <int L>
__device__ __forceinline__ void wait_groups(int u) {
  switch (u) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<L>(); break;
    case 2: wait_vmcnt<2 * L>(); break;
    case 3: wait_vmcnt<3 * L>(); break;
    case 4: wait_vmcnt<4 * L>(); break;
    case 5: wait_vmcnt<5 * L>(); break;
    case 6: wait_vmcnt<6 * L>(); break;
    default: wait_vmcnt<7 * L>(); break;
  }
}

// LDS byte address of a pointer into shared memory.
__device__ __forceinline__ uint32_t lds_addr(const unsigned char* p) {
  return static_cast<uint32_t>((uintptr_t)(lds_void*)p);
}

// Raw buffer resource words over `bytes` bytes at `base` (stride 0, 32-bit
// data): offsets at or past `bytes` read as zero and touch no memory.
__device__ __forceinline__ u32x4 rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  return u32x4{static_cast<uint32_t>(b), static_cast<uint32_t>(b >> 32) & 0xffffu, bytes,
               kRsrcWord3};
}

// 16 bytes per lane from buffer offset voff into LDS at lds_base + 16 * lane
// (buffer_load_dwordx4 ... lds).  Written in assembly so that the compiler does
// not track it: its completion is ordered by explicit waits.  M0 carries the
// LDS base; the compiler keeps no value of its own in M0 in this kernel.
__device__ __forceinline__ void dma16(const u32x4& r, uint32_t lds_base, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(voff), "s"(r), "s"(lds_base)
               : "memory", "m0");
}

// Global loads issued from assembly, like the DMAs: the compiler does not
// track them, so they may overlap the first tile DMAs; the caller waits for
// them with an explicit s_waitcnt and then passes the registers through
// tie_regs() so that no use is scheduled before that wait.
__device__ __forceinline__ u32x4 gload16(const void* p) {
  u32x4 r;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(r) : "v"(p) : "memory");
  return r;
}
__device__ __forceinline__ uint32_t gload4(const void* p) {
  uint32_t r;
  asm volatile("global_load_dword %0, %1, off" : "=v"(r) : "v"(p) : "memory");
  return r;
}
__device__ __forceinline__ u32x2 gload8(const void* p) {
  u32x2 r;
  asm volatile("global_load_dwordx2 %0, %1, off" : "=v"(r) : "v"(p) : "memory");
  return r;
}
template <int N>
__device__ __forceinline__ void tie_regs2(u32x2 (&a)[N], u32x2 (&b)[N], uint32_t& z, uint32_t& e) {
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(a[i]), "+v"(b[i]) : : "memory");
  asm volatile("" : "+v"(z), "+v"(e) : : "memory");
}
template <int N>
__device__ __forceinline__ void tie_regs(u32x4 (&q)[N], uint32_t& z) {
  static_assert(N == 2 || N == 4, "operand count");
  if constexpr (N == 4)
    asm volatile("" : "+v"(q[0]), "+v"(q[1]), "+v"(q[2]), "+v"(q[3]), "+v"(z) : : "memory");
  else
    asm volatile("" : "+v"(q[0]), "+v"(q[1]), "+v"(z) : : "memory");
}

// Workgroup barrier for LDS traffic only: this wave's LDS operations complete,
// then s_barrier.  __syncthreads() would also wait for every outstanding
// vector-memory load; the DMA of the data about to be read is waited for
// explicitly (wait_vmcnt) before this barrier.  The memory clobber keeps the
// compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Weights of one tile in the product's operand layout, and its read mask.
struct TileW {
  u32x4 hi, lo;
  uint64_t mask;
};

template <int D, bool DENSE, bool DBG, bool CX = false, bool EAGER = false, bool F16 = false,
          bool CASC = false, bool LC = true>
__global__ __launch_bounds__(kStkThreads) void decode_stacked_kernel(const DecodeArgs a) {
  constexpr bool PIPE = DENSE || EAGER;  // the dense pipeline: values fetched with their keys
  constexpr bool DEPTH = !DENSE;         // the depth rule decides the weights
  static_assert(!CASC || (PIPE && !DBG && !CX && !F16), "cascade: production BF16 variants");
  constexpr int NK = D / 32;          // K-dim steps of the score product
  constexpr int NB = D / 16;          // 16-channel blocks of the value product
  constexpr int KEYB = 2 * D;         // bytes per key row
  constexpr int CPK = KEYB / 16;      // 16-byte chunks per key row
  constexpr int TILEB = kTile * KEYB; // bytes of one 64-key K (or V) tile
  constexpr int NLD = TILEB / 1024 / kStkWaves;  // 1 KiB DMA loads per wave per tile
  constexpr int KST = 4;              // K stages in LDS
  constexpr int VST = PIPE ? 4 : 3;   // V stages in LDS
  static_assert(D == 64 || D == 128, "head dim");
  static_assert(NLD >= 1 && (NLD * 1024 / KEYB) * kStkWaves == kTile, "tile split");
  static_assert(7 * NLD < 64, "wait counts");
  static_assert(4 * NB * 4 * 64 * 4 + 4 * 64 * 4 <= (KST + VST) * TILEB, "reduction space");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[(KST + VST) * TILEB];
  __shared__ uint32_t gate[kStkWaves];

  const ScanGeometry& g = a.geo;
  const ScanPlace p = scan_place(a);
  if (p.rg * kStkRows >= p.nrows) return;  // uniform: no rows in this read group
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rb = wave & 3;
  const int kh = wave >> 2;
  const int n16 = lane & 15;
  const int grp = lane >> 4;

  const int S = a.num_splits;
  const int ntiles = (p.n + kTile - 1) / kTile;
  const int m_pre = ntiles > p.split ? (ntiles - p.split + S - 1) / S : 0;  // prefix tiles of the split
  // CASC: the suffix tiles of the read group's requests follow the prefix
  // tiles.  Pair q = position * sfx_tiles + tile, over the request positions
  // the group's rows cover, goes to split q mod S; a suffix tile weighs only
  // the rows of its own request (the others get Z = +inf for it).
  int pos_lo = 0, m_sfx = 0;
  if constexpr (CASC) {
    const int r0 = p.rg * kStkRows;
    const int r1 = min(r0 + kStkRows, p.nrows) - 1;
    pos_lo = r0 / g.group;
    const int pairs = (r1 / g.group - pos_lo + 1) * a.sfx_tiles;
    m_sfx = pairs > p.split ? (pairs - p.split + S - 1) / S : 0;
    if (m_pre + m_sfx > kWaveSize) return;  // uniform; the host admits no such call
  }
  const int m = m_pre + m_sfx;  // tiles of this workgroup
  const int my_chunk = wave / 2;  // all of a wave's DMA keys lie in this 16-key chunk of a tile
  auto chunk_of = [&](int j) { return (p.split + j * S) * (kTile / kChunk) + my_chunk; };

  // Block-table entries of this wave's chunk for 64 local tiles, lane j holding
  // tile ptab_base + j; read with v_readlane, reloaded every 64 tiles (callers
  // ask for increasing tiles).
  int ptab = 0;
  int ptab_base = -kWaveSize;
  // CASC: lane j also holds tile j's key count (bits 0-7), the read-group
  // position of its request (bits 8-15; 255 for a prefix tile: every row) and
  // the in-page key offset of this wave's chunk (bits 16-31).  A suffix lane
  // first learns its request (sreq); the request's length and block-table
  // entry follow from assembly loads (slen, sbt) and are merged in settle_sfx.
  uint32_t tmeta = 0;
  int sreq = -1;
  uint32_t slen = 0, sbt = 0;
  auto load_ptab = [&](int base) {
    ptab_base = base;
    const int jj = base + lane;
    const int c = chunk_of(jj);
    if constexpr (CASC) {
      ptab = 0;
      tmeta = 0;
      if (jj < m_pre) {
        // the tile's key count for every wave; the page only where this
        // wave's chunk holds keys
        const int key0 = c * kChunk;
        const int pidx = key0 / g.page_size;
        if (c < p.nchunks) ptab = g.block_table[static_cast<size_t>(p.seq) * g.max_pages + pidx];
        const int t = p.split + jj * S;
        tmeta = static_cast<uint32_t>(min(kTile, p.n - t * kTile)) | (0xFFu << 8) |
                (static_cast<uint32_t>(key0 - pidx * g.page_size) << 16);
      } else if (jj >= m_pre && jj < m) {
        sreq = ld_uniform(g.row_req, p.req0 + pos_lo + (p.split + (jj - m_pre) * S) / a.sfx_tiles);
      }
    } else {
      ptab = jj < m && c < p.nchunks
                 ? g.block_table[static_cast<size_t>(p.seq) * g.max_pages + (c * kChunk) / g.page_size]
                 : 0;
    }
  };
  auto page_of = [&](int j) -> int {
    if (j >= m || g.page_size <= 0) return 0;
    if ((j & ~(kWaveSize - 1)) != ptab_base) {
      load_ptab(j & ~(kWaveSize - 1));
      wait_vmcnt<0>();  // a reload past tile 64: drains the DMAs in flight once
    }
    return __builtin_amdgcn_readlane(ptab, j & (kWaveSize - 1));
  };

  // Prologue loads: the first page-table window and the row list (the
  // compiler waits for both before their values are used), then the row's
  // query and reference from assembly: they are in flight together with the
  // first tile DMAs and have landed once the first key tile has.
  if (g.page_size > 0 && m > 0) load_ptab(0);
  const RowInfo ri = row_info(g, p.seq, p.kvh, p.rg * kStkRows + 16 * rb + n16, p.nrows, p.req0);
  const size_t qrow = static_cast<size_t>(ri.req) * g.heads + ri.head;
  // CASC: a suffix lane's request length and block-table entry, loaded from
  // assembly (a lane without one reads element 0); merged into the tile
  // table once they have landed.
  const int pos_row = (p.rg * kStkRows + 16 * rb + n16) / g.group - pos_lo;
  int u_sfx = 0, pl_sfx = 0;  // this lane's suffix tile and request position
  auto settle_sfx = [&]() {
    if constexpr (CASC) {
      asm volatile("" : "+v"(slen), "+v"(sbt) : : "memory");
      if (lane >= m_pre && lane < m) {
        const int n = sreq >= 0 && sreq < g.batch ? clamp_len(static_cast<int>(slen), a.sfx_cap) : 0;
        const int key0 = u_sfx * kTile + kChunk * my_chunk;
        const int pidx = key0 / g.page_size;
        ptab = key0 < n ? static_cast<int>(sbt) : 0;
        tmeta = static_cast<uint32_t>(max(0, min(kTile, n - u_sfx * kTile))) |
                (static_cast<uint32_t>(pl_sfx) << 8) |
                (static_cast<uint32_t>(key0 - pidx * g.page_size) << 16);
      }
    }
  };
  // Block-table entries of tiles 0..4, read (and the page-table load waited
  // for) before the assembly loads below are issued; the empty asm pins that
  // order.
  int pg0 = page_of(0), pg1 = page_of(1), pg2 = page_of(2), pg3 = page_of(3),
            pg4 = page_of(4);
  asm volatile("" : : "s"(pg0), "s"(pg1), "s"(pg2), "s"(pg3), "s"(pg4));
  if constexpr (CASC) {
    const int32_t* lp = a.sfx_seq_lens;
    const int32_t* bp = a.sfx_block_table;
    if (lane >= m_pre && lane < m) {
      const int qd = p.split + (lane - m_pre) * S;
      pl_sfx = qd / a.sfx_tiles;
      u_sfx = qd - pl_sfx * a.sfx_tiles;
      const int pidx = (u_sfx * kTile + kChunk * my_chunk) / g.page_size;
      if (sreq >= 0 && sreq < g.batch) {
        lp += sreq;
        if (pidx < a.sfx_max_pages) bp += static_cast<size_t>(sreq) * a.sfx_max_pages + pidx;
      }
    }
    slen = gload4(lp);
    sbt = gload4(bp);
    if (m_pre < 5 && m > m_pre) {  // a suffix tile among the first five: wait here
      wait_vmcnt<0>();
      settle_sfx();
      pg0 = page_of(0);
      pg1 = page_of(1);
      pg2 = page_of(2);
      pg3 = page_of(3);
      pg4 = page_of(4);
    }
  }
  u32x4 qb[NK];
  uint32_t zbits;
  // F16 (stacked level of a two-plane key cache): the query codes qa, qb of
  // the lane's channels and the row's score scale eta
  u32x2 qca[F16 ? NK : 1], qcb[F16 ? NK : 1];
  uint32_t ebits = 0;
  {
    // a row outside the group reads row 0 (there is at least one row) and is
    // replaced below
    if constexpr (F16) {
      const int8_t* qp = a.qplanes + (ri.ok ? qrow * 2 * D : 0) + 8 * grp;
#pragma unroll
      for (int c = 0; c < NK; ++c) {
        qca[c] = gload8(qp + 32 * c);
        qcb[c] = gload8(qp + D + 32 * c);
      }
      ebits = gload4(a.qeta + (ri.ok ? qrow : 0));
    } else {
      const uint16_t* qp = a.q + (ri.ok ? qrow * D : 0) + 8 * grp;
#pragma unroll
      for (int c = 0; c < NK; ++c) qb[c] = gload16(qp + 32 * c);
    }
    zbits = gload4(a.z + (ri.ok ? qrow : 0));
  }
  float zr = 0.0f;
  float sscale = a.score_scale;  // F16: the row's eta
  auto settle_row = [&]() {
    if constexpr (F16) {
      tie_regs2(qca, qcb, zbits, ebits);
      // the query operand fp16(qa + qb/256), element k of the 8 at byte k
#pragma unroll
      for (int c = 0; c < NK; ++c) {
        uint32_t h[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const uint32_t wa = k < 4 ? qca[c].x : qca[c].y;
          const uint32_t wb = k < 4 ? qcb[c].x : qcb[c].y;
          const int ca = static_cast<int8_t>((wa >> (8 * (k & 3))) & 0xffu);
          const int cb = static_cast<int8_t>((wb >> (8 * (k & 3))) & 0xffu);
          h[k] = f32_to_f16_bits(static_cast<float>(ca) + static_cast<float>(cb) * (1.0f / 256.0f));
        }
        qb[c] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                      h[6] | (h[7] << 16)};
      }
      sscale = ri.ok ? __uint_as_float(ebits) : 0.0f;
    } else {
      tie_regs(qb, zbits);
    }
    // A row outside the group gets Z = +inf and q = 0: x = -inf, its weights
    // are exactly 0 and it is never live, without per-key selects.
    zr = ri.ok ? __uint_as_float(zbits) : INFINITY;
#pragma unroll
    for (int c = 0; c < NK; ++c) qb[c] = ri.ok ? qb[c] : u32x4{0, 0, 0, 0};
  };

  // Slot permutation of a key row.  With 256-byte rows (D = 128) the 16 keys a
  // K-operand read covers need 16 distinct slots: f = k & 15; the two 16-lane
  // groups of a transposing read cover keys 4i.. and 4i+4.. and take disjoint
  // halves of the row: f = 2 (k & 3) + 8 ((k >> 2) & 1).  With 128-byte rows
  // (D = 64) two keys share a 256-byte bank line: f = (k >> 1) & 7 and
  // f = 2 ((k & 3) ^ ((k >> 2) & 1)).
  auto fk = [](int k) { return D == 128 ? (k & 15) : ((k >> 1) & 7); };
  auto fv = [](int k) {
    return D == 128 ? 2 * (k & 3) + 8 * ((k >> 2) & 1) : 2 * ((k & 3) ^ ((k >> 2) & 1));
  };

  // DMA placement (loop-invariant): load q of this wave fills the 16-byte slots
  // 64 (wave NLD + q) + lane of the tile; slot s of key k receives chunk s ^ f(k).
  uint32_t koff[NLD], voff[NLD];
  int vkey[NLD];
#pragma unroll
  for (int q = 0; q < NLD; ++q) {
    const int slot = 64 * (wave * NLD + q) + lane;
    const int k = slot / CPK;
    const int s = slot % CPK;
    koff[q] = (k % kChunk) * KEYB + ((s ^ fk(k)) << 4);
    voff[q] = (k % kChunk) * KEYB + ((s ^ fv(k)) << 4);
    vkey[q] = k;
  }
  const uint32_t wave_dst = __builtin_amdgcn_readfirstlane(lds_addr(smem) + 1024 * wave * NLD);

  // Buffer resource words of this wave's chunk of local tile j (K or V).
  auto chunk_words = [&](int j, int phys, bool val) -> u32x4 {
    if constexpr (CASC) {
      const uint32_t meta =
          j < m ? static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(tmeta), j)) : 0u;
      const int have = min(kChunk, static_cast<int>(meta & 0xFFu) - kChunk * my_chunk);
      const bool ok = have > 0 && phys >= 0 && phys < g.num_pages;
      const size_t off = ((static_cast<size_t>(ok ? phys : 0) * g.hkv + p.kvh) * g.page_size +
                          (meta >> 16)) * D;
      return rsrc_words((val ? g.v : g.k) + off, ok ? static_cast<uint32_t>(have) * KEYB : 0u);
    }
    const int c = chunk_of(j);
    uint32_t bytes = 0;
    size_t off = 0;
    if (c < p.nchunks) {
      const int key0 = c * kChunk;
      bool ok = true;
      if (g.page_size > 0) {
        const int page = key0 / g.page_size;
        ok = phys >= 0 && phys < g.num_pages;
        off = ((static_cast<size_t>(ok ? phys : 0) * g.hkv + p.kvh) * g.page_size +
               (key0 - page * g.page_size)) * D;
      } else {
        off = ((static_cast<size_t>(p.seq) * g.hkv + p.kvh) * g.max_seq_len + key0) * D;
      }
      if (ok) bytes = static_cast<uint32_t>(min(kChunk, p.n - key0)) * KEYB;
    }
    return rsrc_words((val ? g.v : g.k) + off, bytes);
  };
  auto fetch_k = [&](int j, int phys, int kst) {
    const u32x4 r = chunk_words(j, phys, false);
#pragma unroll
    for (int q = 0; q < NLD; ++q) dma16(r, wave_dst + kst * TILEB + 1024 * q, koff[q]);
  };
  auto fetch_v = [&](int j, int phys, int vst, uint64_t vmask) {
    const u32x4 r = chunk_words(j, phys, true);
#pragma unroll
    for (int q = 0; q < NLD; ++q)
      dma16(r, wave_dst + (KST + vst) * TILEB + 1024 * q,
            ((vmask >> vkey[q]) & 1u) ? voff[q] : kOutOfRange);
  };

  f32x4 acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  float lsum = 0.0f;
  float lcut = 0.0f;  // weights of cut keys (finite depth)

  // S^T of this wave's two 16-key subtiles of the tile in K stage kst.  K
  // operand: lane l reads chunk 4 cc + l/16 of key 32 kh + 16 st + l%16.
  auto qk = [&](int kst, f32x4 (&s)[2]) {
    const unsigned char* kb = smem + kst * TILEB + (32 * kh + n16) * KEYB;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      f32x4 c4 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int cc = 0; cc < NK; ++cc) {
        const u32x4 kop = *reinterpret_cast<const u32x4*>(
            kb + 16 * KEYB * st + (((4 * cc + grp) ^ fk(n16)) << 4));
        c4 = F16 ? mfma_16x16x32_f16(kop, qb[cc], c4) : mfma_16x16x32(kop, qb[cc], c4);
      }
      s[st] = c4;
    }
  };

  // Keys of local tile j that exist (64 for every tile but a split's last
  // partial one; 0 or less past the split's end).
  auto tile_keys = [&](int j) {
    if constexpr (CASC)
      return j < m ? (__builtin_amdgcn_readlane(static_cast<int>(tmeta), j) & 0xFF) : 0;
    return min(kTile, p.n - (p.split + j * S) * kTile);
  };

  // Verdicts, L and the product operands of local tile j from its scores; when
  // `need_mask`, this wave's 32-bit live mask over its key half goes to gate[].
  // FULL: all 64 keys exist (no per-key selects; rows outside the group have
  // x = -inf).  Otherwise keys past the end are selected away, which also keeps
  // a stale K stage (tiles past the split's end) out of the result.
  auto weigh = [&](auto full_tag, int j, const f32x4 (&s)[2], bool need_mask) -> TileW {
    constexpr bool FULL = decltype(full_tag)::value;
    const int key0 = (p.split + j * S) * kTile;
    const int nk = tile_keys(j);
    float zt = zr;  // CASC: +inf for rows outside a suffix tile's request
    if constexpr (CASC) {
      const int code =
          j < m ? ((__builtin_amdgcn_readlane(static_cast<int>(tmeta), j) >> 8) & 0xFF) : 0xFF;
      zt = code == 0xFF || code == pos_row ? zr : INFINITY;
    }
    uint32_t hb[2][4];
    float lf[2][4];
    float cc[2] = {0.0f, 0.0f};  // cut weights of this lane's keys of the half's two chunks
    uint32_t lb = 0;  // bit 4 st + i: key 16 st + 4 grp + i of the half is live for this row
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kk = 32 * kh + 16 * st + 4 * grp + i;
        const bool ok = FULL || (ri.ok && kk < nk);
        const float x = __builtin_fmaf(s[st][i], sscale, -zt);
        const bool live = ok && (!DEPTH || x >= a.neg_T);
        const float w = FULL ? exp2_fast(x) : (ok ? exp2_fast(x) : 0.0f);
        lsum += w;
        if (DEPTH && LC) lcut += live ? 0.0f : w;  // LC: the caller asked for the cut mass
        if (DEPTH && (CX || DBG)) cc[st] += live ? 0.0f : w;
        const float pw = (FULL && !DEPTH) ? w : (live ? w : 0.0f);
        hb[st][i] = __float_as_uint(pw) & 0xffff0000u;
        lf[st][i] = pw - __uint_as_float(hb[st][i]);
        lb |= (live ? 1u : 0u) << (4 * st + i);
        if (DBG && a.x_out && ri.ok && kk < nk) a.x_out[qrow * g.max_seq_len + key0 + kk] = x;
      }
    if constexpr (DEPTH && (CX || DBG)) {
      if (a.chunk_cut) {
        // the four key groups of row n16 hold a chunk's 16 keys
#pragma unroll
        for (int st = 0; st < 2; ++st) {
          float t = cc[st];
          t += __shfl_xor(t, 16, 64);
          t += __shfl_xor(t, 32, 64);
          const int c = (key0 + 32 * kh + 16 * st) / kChunk;
          if (grp == 0 && ri.ok && c < p.nchunks) a.chunk_cut[qrow * a.chunk_stride + c] = t;
        }
      }
    }
    if (need_mask) {
      lb = group_or16(lb);
      uint32_t mask = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t mq = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(lb), 16 * q));
        mask |= ((mq & 0xFu) << (4 * q)) | ((mq & 0xF0u) << (12 + 4 * q));
      }
      if (lane == 0) gate[wave] = mask;
    }
    TileW t;
    t.hi = u32x4{(hb[0][0] >> 16) | hb[0][1], (hb[0][2] >> 16) | hb[0][3],
                 (hb[1][0] >> 16) | hb[1][1], (hb[1][2] >> 16) | hb[1][3]};
    t.lo = u32x4{pack_bf16_rne(lf[0][0], lf[0][1]), pack_bf16_rne(lf[0][2], lf[0][3]),
                 pack_bf16_rne(lf[1][0], lf[1][1]), pack_bf16_rne(lf[1][2], lf[1][3])};
    t.mask = ~0ull;
    return t;
  };

  // A^T += V^T P^T over this wave's 32 keys of the tile in V stage vst.
  // Transposing read: source lane 4i + a of group l/16 points at channels
  // 16 blk + 4a .. +4 of key 4(l/16) + i (+16 for the second read); lane l
  // receives channel 16 blk + l%16 of those four keys.  Chunk c = 2 blk + a/2
  // of key k sits in slot c ^ fv(k), i.e. at byte 32 (blk ^ (fv(k) / 2)) + 8a.
  const int i4 = n16 >> 2;
  const int a4 = n16 & 3;
  const int vsw = fv(4 * grp + i4) >> 1;
  const unsigned char* vlane = smem + KST * TILEB + (32 * kh + 4 * grp + i4) * KEYB + 8 * a4;
  auto product = [&](int vst, const TileW& t) {
    const unsigned char* vb = vlane + vst * TILEB;
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
      const unsigned char* e = vb + 32 * (blk ^ vsw);
      const u32x2 r0 = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)e));
      const u32x2 r1 =
          __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(e + 16 * KEYB)));
      const u32x4 va = {r0.x, r0.y, r1.x, r1.y};
      acc[blk] = mfma_16x16x32(va, t.hi, acc[blk]);
      acc[blk] = mfma_16x16x32(va, t.lo, acc[blk]);
    }
  };

  auto read_gate = [&]() -> uint64_t {
    const uint32_t lo = gate[0] | gate[1] | gate[2] | gate[3];
    const uint32_t hi = gate[4] | gate[5] | gate[6] | gate[7];
    // readfirstlane returns int: go through uint32_t so that bit 31 of the low
    // word does not sign-extend into the high word.
    const uint32_t l = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(lo)));
    const uint32_t h = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(hi)));
    return static_cast<uint64_t>(l) | (static_cast<uint64_t>(h) << 32);
  };

  const size_t gate_row = (static_cast<size_t>(p.seq) * g.hkv + p.kvh) * a.row_groups + p.rg;
  auto debug_gates = [&](int j, uint64_t tm) {
    if (!DBG || wave != 0) return;
    const int key0 = (p.split + j * S) * kTile;
    const int nk = min(kTile, p.n - key0);
    if (a.key_gate_out && lane < nk)
      a.key_gate_out[gate_row * g.max_seq_len + key0 + lane] = (tm >> lane) & 1u;
    if (a.page_gate_out && lane < kTile / kChunk && kChunk * lane < nk)
      a.page_gate_out[gate_row * ((g.max_seq_len + kChunk - 1) / kChunk) + key0 / kChunk + lane] =
          ((tm >> (kChunk * lane)) & 0xffffull) ? 1 : 0;
  };
  auto next_stage = [](int s, int n) { return s == n - 1 ? 0 : s + 1; };

  using Full = std::true_type;
  using Part = std::false_type;

  if (PIPE && m > 0) {
    // Issue order: K0, then pairs (K(i+1), V(i)).  Keys of tile j in K stage
    // j % 4, values in V stage j % 4.
    fetch_k(0, pg0, 0);
    int issued = 0;  // pairs issued
    if (m > 0) { if (m > 1) fetch_k(1, pg1, 1); fetch_v(0, pg0, 0, ~0ull); ++issued; }
    if (m > 1) { if (m > 2) fetch_k(2, pg2, 2); fetch_v(1, pg1, 1, ~0ull); ++issued; }
    if (m > 2) { if (m > 3) fetch_k(3, pg3, 3); fetch_v(2, pg2, 2, ~0ull); ++issued; }
    // K0 landed: behind it two groups per issued pair, less the key group of
    // a pair whose tile i+1 does not exist
    wait_groups<NLD>(2 * issued - (issued == m ? 1 : 0));
    settle_row();  // Q and Z were issued before K0
    if (CASC && m_pre >= 5) settle_sfx();  // so were the suffix lanes' loads
    lds_barrier();
    f32x4 s[2];
    qk(0, s);
    TileW w = tile_keys(0) == kTile ? weigh(Full{}, 0, s, DBG) : weigh(Part{}, 0, s, DBG);
    if (DBG) {
      lds_barrier();
      debug_gates(0, read_gate());
    }
    int ks1 = 1, vs0 = 0, s3 = 3;  // K stage of t+1, V stage of t, stage of tile t+3
    int pv3 = pg3;                  // page of tile t+3 (values)
    int pk4 = pg4;                  // page of tile t+4 (keys)
    for (int t = 0; t < m; ++t) {
      // landed: K(t+1), V(t); in flight behind them: pairs t+1, t+2
      wait_groups<NLD>((t + 2 < m) + (t + 1 < m) + (t + 3 < m) + (t + 2 < m));
      lds_barrier();  // every wave is done with K(t) and V(t-1)
      const int pk5 = page_of(t + 5);
      if (t + 4 < m) fetch_k(t + 4, pk4, next_stage(s3, KST));
      if (t + 3 < m) fetch_v(t + 3, pv3, s3, ~0ull);
      // Tile t+1 is scored even past the split's end (a stale stage then; the
      // partial path selects every key away), so that the product of tile t
      // and the weights of tile t+1 form one block the compiler can interleave.
      f32x4 s1[2];
      qk(ks1, s1);
      if (tile_keys(t + 1) == kTile) {
        product(vs0, w);
        w = weigh(Full{}, t + 1, s1, DBG);
      } else {
        product(vs0, w);
        w = weigh(Part{}, t + 1, s1, DBG);
      }
      if (DBG && t + 1 < m) {
        lds_barrier();
        debug_gates(t + 1, read_gate());
      }
      pv3 = pk4;  // tile t+4 becomes tile (t+1)+3
      pk4 = pk5;
      ks1 = next_stage(ks1, KST);
      vs0 = next_stage(vs0, VST);
      s3 = next_stage(s3, KST);
    }
  } else if (!PIPE && m > 0) {
    // Issue order: K0 K1 V0 K2 V1 | K3 V2 | K4 V3 | ...  Keys of tile j in K
    // stage j % 4, values in V stage j % 3.
    const int ph0 = pg0, ph1 = pg1;
    fetch_k(0, ph0, 0);
    if (m > 1) fetch_k(1, ph1, 1);
    wait_groups<NLD>(m > 1 ? 1 : 0);
    settle_row();  // Q and Z were issued before K0
    lds_barrier();
    f32x4 s[2];
    qk(0, s);
    TileW w0 = tile_keys(0) == kTile ? weigh(Full{}, 0, s, true) : weigh(Part{}, 0, s, true);
    lds_barrier();
    w0.mask = read_gate();
    debug_gates(0, w0.mask);
    fetch_v(0, ph0, 0, w0.mask);
    TileW w1 = {};
    int ph2 = pg2, ph3 = pg3;
    if (m > 2) fetch_k(2, ph2, 2);
    if (m > 1) {
      wait_groups<NLD>(m > 2 ? 2 : 1);  // K1 landed; V0, K2 may fly
      lds_barrier();
      qk(1, s);
      w1 = tile_keys(1) == kTile ? weigh(Full{}, 1, s, true) : weigh(Part{}, 1, s, true);
      lds_barrier();
      w1.mask = read_gate();
      debug_gates(1, w1.mask);
      fetch_v(1, ph1, 1, w1.mask);
    }
    int ks2 = 2, ks3 = 3, vs0 = 0, vs2 = 2;  // K stages of t+2, t+3; V stages of t, t+2
    for (int t = 0; t < m; ++t) {
      // registers: weights of tiles t (w0) and t+1 (w1).  K(t+2) and the older
      // V(t) have landed once at most V(t+1) is outstanding behind them.
      wait_groups<NLD>(t + 1 < m ? 1 : 0);
      lds_barrier();  // A: gate[] and the stages of tile t-1 are free
      const int ph4 = page_of(t + 4);
      if (t + 3 < m) fetch_k(t + 3, ph3, ks3);
      // Tile t+2 is scored even past the split's end (see the dense loop); its
      // product of tile t is skipped when no row of the group is live on this
      // wave's key half.
      f32x4 s2[2];
      qk(ks2, s2);
      const bool any = kh ? (w0.mask >> 32) != 0 : (w0.mask & 0xffffffffull) != 0;
      TileW w2;
      if (tile_keys(t + 2) == kTile) {
        if (any) product(vs0, w0);
        w2 = weigh(Full{}, t + 2, s2, true);
      } else {
        if (any) product(vs0, w0);
        w2 = weigh(Part{}, t + 2, s2, true);
      }
      lds_barrier();  // B: gates of tile t+2 complete
      if (t + 2 < m) {
        w2.mask = read_gate();
        debug_gates(t + 2, w2.mask);
        fetch_v(t + 2, ph2, vs2, w2.mask);
      } else {
        w2.mask = 0;
      }
      w0 = w1;
      w1 = w2;
      ph2 = ph3;
      ph3 = ph4;
      ks2 = next_stage(ks2, KST);
      ks3 = next_stage(ks3, KST);
      vs0 = next_stage(vs0, VST);
      vs2 = next_stage(vs2, VST);
    }
  }

  if (m == 0) {
    wait_vmcnt<0>();
    settle_row();
  }

  // L partials: the four lane groups of a row hold different keys.
  lsum += __shfl_xor(lsum, 16, 64);
  lsum += __shfl_xor(lsum, 32, 64);
  if (DEPTH) {
    lcut += __shfl_xor(lcut, 16, 64);
    lcut += __shfl_xor(lcut, 32, 64);
  }

  // Key half 1 hands its partials to key half 0 through LDS (the tiles are dead).
  wait_vmcnt<0>();
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);  // [4 row blocks][NB][4][64]
  float* redl = red + 4 * NB * 4 * 64;          // [4][64]: L (lanes 0-15), cut mass (16-31)
  if (kh == 1) {
#pragma unroll
    for (int blk = 0; blk < NB; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[((rb * NB + blk) * 4 + i) * 64 + lane] = acc[blk][i];
    redl[rb * 64 + lane] = lane < 16 ? lsum : lcut;
  }
  __syncthreads();
  if (kh == 0 && ri.ok) {
    const size_t slot = static_cast<size_t>(a.slot_offset) + p.split;
    const size_t prow = (slot * g.batch + ri.req) * g.heads + ri.head;
    float* dst = a.part_A + prow * D + 4 * grp;
    const bool aligned = (reinterpret_cast<uintptr_t>(a.part_A) & 15) == 0;  // uniform
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
      f32x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = acc[blk][i] + red[((rb * NB + blk) * 4 + i) * 64 + lane];
      if (aligned) {
        *reinterpret_cast<f32x4*>(dst + 16 * blk) = v;
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) dst[16 * blk + i] = v[i];
      }
    }
    if (grp == 0) a.part_L[prow] = lsum + redl[rb * 64 + lane];
    if (grp == 1 && a.part_Lcut) a.part_Lcut[prow] = lcut + redl[rb * 64 + lane];
  }
}

template <int D, bool DENSE, bool F16>
hipError_t launch_stk(const DecodeArgs& a, bool dbg, unsigned blocks, hipStream_t stream) {
  if (dbg) {
    hipLaunchKernelGGL((decode_stacked_kernel<D, DENSE, true, false, false, F16>), dim3(blocks),
                       dim3(kStkThreads), 0, stream, a);
  } else if constexpr (DENSE) {
    hipLaunchKernelGGL((decode_stacked_kernel<D, true, false, false, false, F16>), dim3(blocks),
                       dim3(kStkThreads), 0, stream, a);
  } else if (!F16 && a.chunk_cut) {
    if constexpr (!F16)
      hipLaunchKernelGGL((decode_stacked_kernel<D, false, false, true, true>), dim3(blocks),
                         dim3(kStkThreads), 0, stream, a);
  } else if (a.part_Lcut) {
    hipLaunchKernelGGL((decode_stacked_kernel<D, false, false, false, true, F16>), dim3(blocks),
                       dim3(kStkThreads), 0, stream, a);
  } else {  // no cut mass wanted: the depth rule only selects the weights
    hipLaunchKernelGGL((decode_stacked_kernel<D, false, false, false, true, F16, false, false>),
                       dim3(blocks), dim3(kStkThreads), 0, stream, a);
  }
  return hipGetLastError();
}

template <int D>
hipError_t launch_stk_d(const DecodeArgs& a, bool dbg, unsigned blocks, hipStream_t stream) {
  if (a.qplanes)
    return a.dense ? launch_stk<D, true, true>(a, dbg, blocks, stream)
                   : launch_stk<D, false, true>(a, dbg, blocks, stream);
  return a.dense ? launch_stk<D, true, false>(a, dbg, blocks, stream)
                 : launch_stk<D, false, false>(a, dbg, blocks, stream);
}

template <int D>
hipError_t launch_casc(const DecodeArgs& a, unsigned blocks, hipStream_t stream) {
  if (a.dense)
    hipLaunchKernelGGL((decode_stacked_kernel<D, true, false, false, false, false, true>),
                       dim3(blocks), dim3(kStkThreads), 0, stream, a);
  else if (a.part_Lcut)
    hipLaunchKernelGGL((decode_stacked_kernel<D, false, false, false, true, false, true>),
                       dim3(blocks), dim3(kStkThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((decode_stacked_kernel<D, false, false, false, true, false, true, false>),
                       dim3(blocks), dim3(kStkThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_cascade(const DecodeArgs& a, int head_dim, hipStream_t stream) {
  if (a.rows_per_group != kStkRows || a.qplanes || a.x_out || a.key_gate_out ||
      a.page_gate_out || a.chunk_cut || a.geo.page_size <= 0 || a.sfx_tiles < 1)
    return hipErrorInvalidValue;
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv * a.num_splits *
                           a.row_groups;
  if (blocks == 0) return hipSuccess;
  const unsigned nb = static_cast<unsigned>(blocks);
  if (head_dim == 128) return launch_casc<128>(a, nb, stream);
  if (head_dim == 64) return launch_casc<64>(a, nb, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_decode_stacked(const DecodeArgs& a, int head_dim, hipStream_t stream) {
  if (a.rows_per_group != kStkRows) return hipErrorInvalidValue;
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv * a.num_splits *
                           a.row_groups;
  if (blocks == 0) return hipSuccess;
  const bool dbg = a.x_out || a.key_gate_out || a.page_gate_out;
  const unsigned nb = static_cast<unsigned>(blocks);
  if (head_dim == 128) return launch_stk_d<128>(a, dbg, nb, stream);
  if (head_dim == 64) return launch_stk_d<64>(a, dbg, nb, stream);
  return hipErrorInvalidValue;
}

}  // namespace fold
