// gfx950 kernels of the owner-scoped fast-weight READ/WRITE path.
//
// READ  (ApplyState, Section 3 "Read"):   y_r = x_r W0 + x_r dW_r
// WRITE (BoundaryUpdate, Section 3 "Write"): shadow_r = live_r + eta Z_r^T G_r
//
// Both operate on groups of owners, one launch per (group, layer).

#include <algorithm>
#include <mutex>

#include "rwttt_kernels.h"

namespace rwttt {
namespace {

#include "rwttt_device.h"

// ---------------------------------------------------------------------------
// READ
// ---------------------------------------------------------------------------
//
// y_b = x_b W0 + x_b dW_b, as two launches with no cross-block
// synchronisation:
//
// 1. read_partial_kernel: one 256-thread block per (group slot b, K chunk of
//    256 rows, column tile).  Each lane owns 16 contiguous bytes of every dW_b
//    row of the tile (4 fp32 or 8 bf16 columns) and the same columns of W0;
//    the four waves split the chunk's rows.  Per row it accumulates
//    x[k]*dW[k] and then x[k]*W0[k] into one fp32 accumulator, so the shared
//    W0 term is fused into the same pass.  The W0 tile is the same for every
//    slot: the blocks of all slots for one (chunk, tile) are placed on one XCD
//    (dispatch is round-robin over the 8 XCDs by block index) so that W0 comes
//    from HBM once and is re-read from that XCD's L2.  Which XCD takes a pair
//    rotates with the pair's round of eight: with 10 column tiles a fixed
//    pair % 8 gave the even XCDs only even tiles, whose blocks ran ~7% slower
//    than the odd tiles' (3% once every XCD mixes both: an address effect,
//    not an XCD one), so those XCDs finished last.  dW is streamed with
//    non-temporal loads so it does not evict W0.  The four waves' sums are
//    added through LDS in a fixed order into one partial per (owner, chunk).
// 2. read_reduce_kernel: y[b, n] = sum over chunks: four contiguous quarters
//    of the chunks, each in chunk order, added in order.
//
// Partials are indexed by owner id, so concurrent reads of disjoint owner sets
// (one per stream) never touch the same workspace bytes.
//
// Every order depends only on the matrix shape, so an owner's y is
// bit-identical whatever the group's size, order or other members.

struct ReadParams {
  const void* x;
  void* y;
  const void* w0;
  float* part;
  int count, d_ff, d_model, ks, nt, npad;
  int slot_part;             // partial sums indexed by group slot (1) or by owner id (0)
  const void* dw[RWTTT_MAX_GROUP];
  uint32_t row[RWTTT_MAX_GROUP];
  void* tail[RWTTT_MAX_GROUP];     // TailBufferUpdate: row receiving x, or null
};

constexpr int kUnroll = 8;

template <typename IO, typename ST>
__global__ void __launch_bounds__(kReadThreads) read_partial_kernel(const ReadParams p) {
  constexpr int COLS = 16 / sizeof(ST);
  constexpr int TILE_N = 64 * COLS;
  constexpr int KC = kReadChunk;
  constexpr int RW = KC / 4;
  __shared__ float xs[KC];
  __shared__ float red[4][TILE_N];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  // block -> (XCD, position on that XCD) -> ((chunk, tile) pair, slot).  Round
  // pl of eight pairs is dealt to the XCDs rotated by pl, so that each XCD
  // gets column tiles of both parities even when the tile count is even
  const int xcd = blockIdx.x & 7;
  const int pos = blockIdx.x >> 3;
  const int pl = pos / p.count;
  const int b = pos - pl * p.count;
  const int pair = pl * 8 + ((xcd + pl) & 7);
  if (pair >= p.ks * p.nt) return;
  const int kc = pair / p.nt;
  const int nt = pair - kc * p.nt;
  const int k0 = kc * KC;
  const int kn = min(KC, p.d_ff - k0);
  const int col = nt * TILE_N + lane * COLS;
  const bool col_ok = col < p.d_model;

  for (int k = tid; k < KC; k += kReadThreads)
    xs[k] = k < kn ? Elem<IO>::get(p.x, size_t(p.row[b]) * p.d_ff + k0 + k) : 0.f;
  if (p.tail[b] != nullptr && nt == 0) {
    // TailBufferUpdate: the first column tile's blocks append this chunk of x
    const IO* xr = static_cast<const IO*>(p.x) + size_t(p.row[b]) * p.d_ff + k0;
    IO* tr = static_cast<IO*>(p.tail[b]) + k0;
    for (int k = tid; k < kn; k += kReadThreads) tr[k] = xr[k];
  }
  __syncthreads();

  const int kw0 = wave * RW;
  const int kw1 = min(kw0 + RW, kn);
  float acc[COLS];
#pragma unroll
  for (int c = 0; c < COLS; ++c) acc[c] = 0.f;
  if (col_ok) {
    const ST* dbase = static_cast<const ST*>(p.dw[b]) + size_t(k0) * p.d_model + col;
    const IO* wbase = static_cast<const IO*>(p.w0) + size_t(k0) * p.d_model + col;
    for (int k = kw0; k < kw1; k += kUnroll) {
      Packed<ST, COLS> v[kUnroll];
      Packed<IO, COLS> w[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        if (k + u < kw1) {
          load_packed<true>(dbase + size_t(k + u) * p.d_model, v[u]);
          load_packed<false>(wbase + size_t(k + u) * p.d_model, w[u]);
        } else {
          v[u].zero();
          w[u].zero();
        }
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const float xv = xs[k + u];
#pragma unroll
        for (int c = 0; c < COLS; ++c) acc[c] = fmaf(xv, w[u].get(c), fmaf(xv, v[u].get(c), acc[c]));
      }
    }
  }
#pragma unroll
  for (int c = 0; c < COLS; ++c) red[wave][lane * COLS + c] = acc[c];
  __syncthreads();
  const uint32_t prow = p.slot_part ? uint32_t(b) : p.row[b];
  float* dst = p.part + (size_t(prow) * p.ks + kc) * p.npad + nt * TILE_N;
  for (int j = tid; j < TILE_N; j += kReadThreads)
    dst[j] = ((red[0][j] + red[1][j]) + red[2][j]) + red[3][j];
}

// 64 output columns per block; the four waves each add a contiguous quarter of
// the chunks in chunk order with all of its loads in flight at once, and the
// quarters are added in order.
constexpr int kRedCols = 64;
constexpr int kRedBatch = 16;

template <typename IO>
__global__ void __launch_bounds__(256) read_reduce_kernel(const ReadParams p) {
  __shared__ float qs[4][kRedCols];
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = blockIdx.x * kRedCols + lane;
  const int per = (p.ks + 3) / 4;
  const int k0 = wave * per, k1 = min(p.ks, k0 + per);
  float s = 0.f;
  if (n < p.d_model) {
    const uint32_t prow = p.slot_part ? uint32_t(b) : p.row[b];
    const float* q = p.part + size_t(prow) * p.ks * p.npad + n;
    for (int k = k0; k < k1; k += kRedBatch) {
      float a[kRedBatch];
#pragma unroll
      for (int u = 0; u < kRedBatch; ++u) a[u] = k + u < k1 ? q[size_t(k + u) * p.npad] : 0.f;
#pragma unroll
      for (int u = 0; u < kRedBatch; ++u) s += a[u];
    }
  }
  qs[wave][lane] = s;
  __syncthreads();
  if (wave == 0 && n < p.d_model)
    Elem<IO>::put(p.y, size_t(p.row[b]) * p.d_model + n, ((qs[0][lane] + qs[1][lane]) + qs[2][lane]) + qs[3][lane]);
}

// ---------------------------------------------------------------------------
// WRITE: shadow = live + eta Z^T G
// ---------------------------------------------------------------------------

struct WriteParams {
  int count, chunk, d_ff, d_model, mt, ntl;
  int parts, npadw;          // streaming path: row-tile partitions per owner; token partial pitch
  float eta;
  const void* x;             // fused token: [n_owners, d_ff] owner-indexed inputs, or null
  const void* w0;            // fused token: W0 of the layer
  float* tpart;              // fused token: [n_owners][parts][npadw] partial sums
  const void* live[RWTTT_MAX_GROUP];
  void* shadow[RWTTT_MAX_GROUP];
  const void* z[RWTTT_MAX_GROUP];
  const void* g[RWTTT_MAX_GROUP];
  uint32_t row[RWTTT_MAX_GROUP];   // owner id of each group slot
};

// ---------------------------------------------------------------------------
// WRITE, bf16 evidence, small chunk (C <= 64): streaming rank-C update
// ---------------------------------------------------------------------------
//
// For C <= 64 the update moves 2 x |dW| bytes for only 2C flop per element,
// so it is HBM-bound and must stream like a copy: what matters is how many
// bytes each CU keeps in flight.  Each block owns one (group slot, 256-column
// tile, partition) and walks the partition's 32-row items (row tiles part,
// part + P, part + 2P, ...; P fixed by the shape).  The owner's G tile is
// staged once per block into LDS, transposed to rank-contiguous rows.  Per
// item, everything the next item needs from HBM (its live rows, its Z tile,
// and for the token its W0 rows and x values) is requested first; then Z's
// 32 x C tile goes through LDS to rank-contiguous rows, the MFMAs form
// D[m][n] = sum_c Z[c][m] G[c][n], the accumulators go through LDS, and every
// wave reads, updates and stores whole 1 KB rows of the slot.  No load is on
// the critical path of the item that issues it.
//
// With a fused token (the WRITE step's own output, read at version v before
// the candidate is committed) the block also loads the same rows of W0 and
// accumulates x[m] * live[m] + x[m] * W0[m] over its items: the live state is
// read once for both the token and the update.  Per-(owner, partition)
// partials are reduced in partition order by read_reduce_kernel.  The blocks
// of all slots for one (tile, partition) sit on one XCD so that W0 comes from
// HBM once.  The partition of an owner's rows never depends on the group, so
// an owner's token and candidate are bit-identical in any group.

constexpr int kSTM = 32;                 // rows per item
constexpr int kSTN = 256;                // columns per tile
constexpr int kSMaxC = 64;               // largest chunk on this path
constexpr int kSPitch = kSMaxC + 8;      // bf16 per staged rank row (144 B: 16 rows hit 16 bank groups)
constexpr int kSParts = 64;              // most row-tile partitions per (owner, column tile)
constexpr int kSSlots = 512;             // blocks of this kernel resident at once (256 CUs x 2)

// Row-tile partitions per (owner, column tile), from the shape alone, so that
// an owner's token partials are added in the same order in any group: as many
// as let one owner's blocks fill one round of the block slots, then the fewest
// that keep the largest partition at the same number of items.
int stream_parts(int d_ff, int d_model) {
  const int mt = (d_ff + kSTM - 1) / kSTM;
  const int ntl = (d_model + kSTN - 1) / kSTN;
  const int pmax = std::max(1, std::min(std::min(kSParts, mt), kSSlots / ntl));
  const int items = (mt + pmax - 1) / pmax;
  return (mt + items - 1) / items;
}

// Rows m0 + 8 wave .. + 7 of a [d_ff, d_model] matrix, 4 columns at ncol.  The
// live state is read once (non-temporal); W0 is read by every slot of the
// group from the same XCD and must stay in its L2 (NT = false).
template <bool NT = true, typename T>
__device__ __forceinline__ void stream_load_rows(const T* base, int d_ff, int d_model, int m0,
                                                 int wave, int ncol, bool ncol_ok,
                                                 Packed<T, 4> (&v)[kSTM / 4]) {
#pragma unroll
  for (int rr = 0; rr < kSTM / 4; ++rr) {
    const int m = m0 + wave * (kSTM / 4) + rr;
    if (m < d_ff && ncol_ok) load_packed<NT>(base + size_t(m) * d_model + ncol, v[rr]);
    else v[rr].zero();
  }
}

// Ranks 2cp, 2cp+1 of eight consecutive rows starting at r0 of a rank-major
// [C][ld] bf16 matrix (threads 0..127: cp = tid / 4, rows r0 + 8 (tid % 4)).
__device__ __forceinline__ void stream_load_pair(const uint16_t* M, int ld, int rows, int chunk,
                                                 int r0, int tid, uint4& a, uint4& b) {
  a = make_uint4(0, 0, 0, 0);
  b = make_uint4(0, 0, 0, 0);
  const int cp = tid >> 2, r = r0 + (tid & 3) * 8, c = 2 * cp;
  if (tid < 128 && r < rows) {
    if (c < chunk) a = *reinterpret_cast<const uint4*>(M + size_t(c) * ld + r);
    if (c + 1 < chunk) b = *reinterpret_cast<const uint4*>(M + size_t(c + 1) * ld + r);
  }
}

// ...and their transpose into rank-contiguous LDS rows dst[row][rank].
__device__ __forceinline__ void stream_store_pair(uint16_t* dst, int tid, int row0, uint4 a,
                                                  uint4 b) {
  if (tid >= 128) return;
  const int cp = tid >> 2, r = row0 + (tid & 3) * 8;
  const uint32_t x[4] = {a.x, a.y, a.z, a.w}, y[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    *reinterpret_cast<uint32_t*>(&dst[(r + 2 * q) * kSPitch + 2 * cp]) = (x[q] & 0xffffu) | (y[q] << 16);
    *reinterpret_cast<uint32_t*>(&dst[(r + 2 * q + 1) * kSPitch + 2 * cp]) = (x[q] >> 16) | (y[q] & 0xffff0000u);
  }
}

template <typename ST, bool TOKEN>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
write_stream_kernel(const WriteParams p) {
  constexpr int RPW = kSTM / 4;           // epilogue rows per wave
  constexpr int KSMAX = kSMaxC / 16;      // MFMA k-steps
  __shared__ __attribute__((aligned(16))) uint16_t zt[kSTM * kSPitch];
  __shared__ __attribute__((aligned(16))) uint16_t gt[kSTN * kSPitch];
  __shared__ __attribute__((aligned(16))) float out[kSTM * kSTN];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int half = lane >> 5;
  // block -> (XCD, position) -> ((tile, partition) pair, slot)
  const int xcd = blockIdx.x & 7;
  const int pos = blockIdx.x >> 3;
  const int pl = pos / p.count;
  const int b = pos - pl * p.count;
  const int pair = pl * 8 + xcd;
  if (pair >= p.ntl * p.parts) return;
  const int nt = pair / p.parts;
  const int part = pair - nt * p.parts;   // parts <= mt: every partition has an item
  const int n0 = nt * kSTN;
  const int ncol = n0 + lane * 4;
  const bool ncol_ok = ncol < p.d_model;
  const int ksteps = (p.chunk + 15) / 16;
  const float eta = p.eta;
  const ST* live = static_cast<const ST*>(p.live[b]);
  ST* shadow = static_cast<ST*>(p.shadow[b]);
  const uint16_t* Z = static_cast<const uint16_t*>(p.z[b]);
  const uint16_t* G = static_cast<const uint16_t*>(p.g[b]);
  const uint16_t* W0 = static_cast<const uint16_t*>(p.w0);
  const uint16_t* X = static_cast<const uint16_t*>(p.x) + size_t(p.row[b]) * p.d_ff;

  // G tile [C ranks][256 n] -> gt[n][rank], 32 columns per thread pass.
  // Every G request and every request of the first item goes out before
  // any of them is used, so the block's start costs one memory round trip
  // (each use of a value loaded under a lane condition waits for all
  // outstanding loads).
  uint4 ga[kSTN / 32], gb[kSTN / 32];
#pragma unroll
  for (int j = 0; j < kSTN / 32; ++j)
    stream_load_pair(G, p.d_model, p.d_model, p.chunk, n0 + j * 32, tid, ga[j], gb[j]);

  // the first item's operands
  float yacc[4] = {0.f, 0.f, 0.f, 0.f};
  Packed<ST, 4> lv[RPW];
  Packed<uint16_t, 4> wv[RPW];
  uint4 za, zb, xq = make_uint4(0, 0, 0, 0);
  stream_load_rows(live, p.d_ff, p.d_model, part * kSTM, wave, ncol, ncol_ok, lv);
  stream_load_pair(Z, p.d_ff, p.d_ff, p.chunk, part * kSTM, tid, za, zb);
  if (TOKEN) {
    stream_load_rows<false>(W0, p.d_ff, p.d_model, part * kSTM, wave, ncol, ncol_ok, wv);
    if (part * kSTM + wave * RPW < p.d_ff)
      xq = *reinterpret_cast<const uint4*>(X + part * kSTM + wave * RPW);
  }
#pragma unroll
  for (int j = 0; j < kSTN / 32; ++j) stream_store_pair(gt, tid, j * 32, ga[j], gb[j]);

  for (int mt = part; mt < p.mt; mt += p.parts) {
    const int m0 = mt * kSTM;
    const int mn = mt + p.parts;
    stream_store_pair(zt, tid, 0, za, zb);
    __syncthreads();
    // the next item's operands load while this one is computed and stored
    Packed<ST, 4> nx[RPW];
    Packed<uint16_t, 4> nw[RPW];
    uint4 nxq = make_uint4(0, 0, 0, 0);
    if (mn < p.mt) {
      stream_load_rows(live, p.d_ff, p.d_model, mn * kSTM, wave, ncol, ncol_ok, nx);
      stream_load_pair(Z, p.d_ff, p.d_ff, p.chunk, mn * kSTM, tid, za, zb);
      if (TOKEN) {
        stream_load_rows<false>(W0, p.d_ff, p.d_model, mn * kSTM, wave, ncol, ncol_ok, nw);
        if (mn * kSTM + wave * RPW < p.d_ff)
          nxq = *reinterpret_cast<const uint4*>(X + mn * kSTM + wave * RPW);
      }
    }
    f32x16_t acc[2] = {f32x16_t{}, f32x16_t{}};
#pragma unroll
    for (int s = 0; s < KSMAX; ++s) {
      if (s < ksteps) {
        const int kofs = s * 16 + half * 8;
        const bf16x8_t az = *reinterpret_cast<const bf16x8_t*>(&zt[(lane & 31) * kSPitch + kofs]);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const bf16x8_t bg = *reinterpret_cast<const bf16x8_t*>(
              &gt[((wave * 2 + i) * 32 + (lane & 31)) * kSPitch + kofs]);
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(az, bg, acc[i], 0, 0, 0);
        }
      }
    }
    // accumulator register 4q+e of lane l holds D[8q + 4(l/32) + e][l % 32]
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        out[(8 * (r >> 2) + 4 * half + (r & 3)) * kSTN + (wave * 2 + i) * 32 + (lane & 31)] = acc[i][r];
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr) {
      const int row = wave * RPW + rr;
      const int m = m0 + row;
      if (m < p.d_ff && ncol_ok) {
        float o[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) o[c] = lv[rr].get(c) + eta * out[row * kSTN + lane * 4 + c];
        store_n<4, true>(shadow + size_t(m) * p.d_model + ncol, o);
      }
    }
    if (TOKEN) {
      // token: x[m] * live[m] + x[m] * W0[m] over this wave's rows, in row order
      const uint32_t xw[4] = {xq.x, xq.y, xq.z, xq.w};
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr) {
        const float xv = (rr & 1) ? bf16_hi(xw[rr >> 1]) : bf16_lo(xw[rr >> 1]);
#pragma unroll
        for (int c = 0; c < 4; ++c) yacc[c] = fmaf(xv, wv[rr].get(c), fmaf(xv, lv[rr].get(c), yacc[c]));
      }
    }
    if (mn < p.mt) {
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr) {
        lv[rr] = nx[rr];
        if (TOKEN) wv[rr] = nw[rr];
      }
      xq = nxq;
    }
    __syncthreads();
  }

  if (TOKEN) {
    // the four waves' token sums in wave order -> one partial per (owner, partition)
#pragma unroll
    for (int c = 0; c < 4; ++c) out[wave * kSTN + lane * 4 + c] = yacc[c];
    __syncthreads();
    const float v = ((out[tid] + out[kSTN + tid]) + out[2 * kSTN + tid]) + out[3 * kSTN + tid];
    p.tpart[(size_t(p.row[b]) * p.parts + part) * p.npadw + n0 + tid] = v;
  }
}

// ---------------------------------------------------------------------------
// WRITE, bf16 evidence, large chunk (C > 64): tiled GEMM
// ---------------------------------------------------------------------------
//
// At C = 512 the update does 2C flop per state element and is near the MFMA
// ridge, so it is organised as a GEMM: D = Z^T G per 256-row (d_ff) x
// 128-column (d_model) tile, four waves of 64 x 128 (2 x 4 MFMA 32x32x16
// blocks, 128 accumulators per lane), two blocks per CU.  The two blocks of
// a CU run independently, so one block's HBM-bound epilogue (read live,
// write shadow) overlaps the other's MFMA main loop.
//
// Operand staging uses no registers: Z and G arrive rank-major and are
// copied as they are, 16 bytes per lane, by buffer loads that write LDS
// directly (lane l of a load lands at LDS offset 16 l).  Ranks are consumed
// in stages of 32 (A: 32 x 256 of Z, B: 32 x 128 of G, 24 KB), three stages
// in flight; each wait names how many newer copies may still be
// outstanding.  The buffer range check turns every 16-byte group outside the
// chunk or the matrix into zeros, so ragged tiles need no other code.  The
// MFMA operands (8 consecutive ranks of one row m or column n) are read back
// with the transposing LDS read ds_read_b64_tr_b16: within each 16-lane
// group, lane i receives element i % 4 of the 8-byte runs addressed by lanes
// 4j + i / 4, so lanes 4j + q address rank row j, columns 4q..4q+3 and two
// such reads give one operand.  The 16-byte groups of rank row r sit in slot
// (group ^ swz(r & 3)), swz = {0, 10, 4, 14}, chosen so that every
// transposing read is free of bank conflicts.
//
// The MFMA is issued as D^T = G^T Z, so the accumulators of a lane hold runs
// of four consecutive columns of one state row.  The epilogue combines them
// with the live rows in that layout (bf16 state: live copied non-temporally
// into the freed stages; fp32 state: a register epilogue through a private LDS region) and
// stores whole rows, rounding to bf16 with the hardware packed convert.

constexpr int kGTM = 256;                                 // rows (d_ff) per tile
constexpr int kGTN = 128;                                 // columns (d_model) per tile
constexpr int kGKC = 32;                                  // ranks per LDS stage
constexpr int kGThreads = 256;                            // 4 waves of 64 x 128
constexpr int kGStageA = kGKC * kGTM;                     // bf16 elements of Z per stage
constexpr int kGStage = kGStageA + kGKC * kGTN;           // 24 KB per stage
constexpr int kGUnitsA = kGStageA * 2 / 1024;             // 1 KB copies of Z per stage (16)
constexpr int kGUnits = kGStage * 2 / 1024;               // 1 KB copies per stage (24)
constexpr int kGCopies = kGUnits / 4;                     // copies per wave per stage (6)
constexpr int kGColGroups = 2;                            // column-tile groups over the XCDs
constexpr int kGRowClasses = 8 / kGColGroups;             // row-tile classes over the XCDs

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

__device__ __forceinline__ int gemm_swz(int r) { return ((r & 3) * 2) ^ ((r & 1) << 3); }

// s_waitcnt with vmcnt(N) and lgkmcnt(0), expcnt left open; no memory access
// moves across it
template <int N>
__device__ __forceinline__ void gemm_wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ void gemm_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

typedef short i16x8_t __attribute__((ext_vector_type(8)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));

// Buffer descriptor of `bytes` bytes at p: no stride, 32-bit data format
// (accesses at or past `bytes` return zeros and touch no memory).
__device__ __forceinline__ i32x4_t gemm_rsrc(const void* p, int bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  return i32x4_t{int(uint32_t(a)), int(uint32_t(a >> 32) & 0xffffu), bytes, 0x00020000};
}

// One 1 KB stage copy: lane l's 16 bytes at byte offset voff of the buffer go
// to LDS at dst + 16 l.  Issued as inline assembly so that the compiler does
// not add its own (conservative) waits for LDS copies: every read of a stage
// is preceded by an explicit vmcnt wait and a barrier.  NT marks the data as
// streamed once (the live state), so that it does not displace the operand
// tiles that the XCD's other blocks still read from L2.
template <bool NT = false>
__device__ __forceinline__ void gemm_copy(uint16_t* dst, uint32_t voff, i32x4_t rsrc) {
  const uint32_t lds = uint32_t(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint16_t*)dst));
  // the descriptor and the LDS address are wave-uniform: keep them in SGPRs
  const i32x4_t r = {__builtin_amdgcn_readfirstlane(rsrc[0]), __builtin_amdgcn_readfirstlane(rsrc[1]),
                     __builtin_amdgcn_readfirstlane(rsrc[2]), __builtin_amdgcn_readfirstlane(rsrc[3])};
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(r) : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(r) : "memory", "m0");
#pragma clang diagnostic pop
}

// One MFMA operand: 8 consecutive ranks (two transposing reads, 4 rank rows
// apart) of the row or column that this lane owns; ROW = LDS row length.
template <int ROW>
__device__ __forceinline__ bf16x8_t gemm_operand(const uint16_t* lds, int off) {
  const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(lds + off));
  const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(lds + off + 4 * ROW));
  return __builtin_bit_cast(bf16x8_t, i16x8_t(__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7)));
}

template <typename ST>
__global__ void __launch_bounds__(kGThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
write_gemm_kernel(const WriteParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t s0[kGStage];
  __shared__ __attribute__((aligned(16))) uint16_t s1[kGStage];
  __shared__ __attribute__((aligned(16))) uint16_t s2[kGStage];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // block -> (owner, row tile, column tile).  Blocks are dealt to the 8
  // XCDs round-robin; XCD x takes column-tile half x % 2 and the row tiles
  // congruent to x / 2 mod 4, so each Z row tile is read by two XCDs and each
  // G column tile by four.  Consecutive blocks of an XCD share their Z row
  // tile, and the XCD's G columns (2 MB at C = 512) stay in its L2 while the
  // live state streams past them non-temporally.
  const int xcd = blockIdx.x & 7;
  const int pos = blockIdx.x >> 3;
  const int ntg = (p.ntl + kGColGroups - 1) / kGColGroups;
  const int mtq = (p.mt + kGRowClasses - 1) / kGRowClasses;
  const int nt = (xcd % kGColGroups) * ntg + pos % ntg;
  const int rest = pos / ntg;
  const int b = rest / mtq;
  const int mt = (rest - b * mtq) * kGRowClasses + xcd / kGColGroups;
  if (nt >= p.ntl || mt >= p.mt || b >= p.count) return;
  const int m0 = mt * kGTM;
  const int n0 = nt * kGTN;
  const uint16_t* Z = static_cast<const uint16_t*>(p.z[b]);
  const uint16_t* G = static_cast<const uint16_t*>(p.g[b]);

  // Stage copies: wave w moves the 1 KB units w, w + 4, w + 8, w + 12 of Z
  // (rank rows 2u, 2u + 1) and w, w + 4 of G (rank rows 4u .. 4u + 3).  Lane
  // l's 16 bytes land at unit offset 16 l, i.e. rank row r, slot s, which
  // holds column group s ^ swz(r).  Byte offsets are relative to the stage's
  // first rank row; a group outside the matrix gets an offset past any range.
  uint32_t voff[kGCopies];
#pragma unroll
  for (int t = 0; t < kGCopies; ++t) {
    const bool za = t < kGUnitsA / 4;
    const int u = wave + 4 * (za ? t : t - kGUnitsA / 4);
    const int r = za ? 2 * u + (lane >> 5) : 4 * u + (lane >> 4);
    const int s = za ? (lane & 31) : (lane & 15);
    const int col = (za ? m0 : n0) + 8 * (s ^ gemm_swz(r));
    const int lim = za ? p.d_ff : p.d_model;
    voff[t] = col < lim ? uint32_t(r * lim + col) * 2u : 0x80000000u;
  }
  auto issue = [&](uint16_t* st, int c0) {
    // rank rows past the chunk fall outside the stage's range: zeros
    const int rows = min(kGKC, p.chunk - c0);
    const i32x4_t zr = gemm_rsrc(Z + size_t(c0) * p.d_ff, rows * p.d_ff * 2);
    const i32x4_t gr = gemm_rsrc(G + size_t(c0) * p.d_model, rows * p.d_model * 2);
#pragma unroll
    for (int t = 0; t < kGCopies; ++t) {
      const bool za = t < kGUnitsA / 4;
      const int u = wave + 4 * (za ? t : t - kGUnitsA / 4);
      gemm_copy(st + (za ? 0 : kGStageA) + u * 512, voff[t], za ? zr : gr);
    }
  };

  // operand read offsets (elements, stage-relative) of this lane's fragments
  const int g4 = lane >> 4;
  const int eps = g4 & 1;
  const int hh = g4 >> 1;
  const int jrow = (lane & 15) >> 2;
  const int q = lane & 3;
  const int sw = gemm_swz(jrow);
  int offa[2], offb[4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
    offa[i] = (8 * hh + jrow) * kGTM + 4 * (q & 1) + (((wave * 8 + i * 4 + 2 * eps + (q >> 1)) ^ sw) << 3);
#pragma unroll
  for (int j = 0; j < 4; ++j)
    offb[j] = kGStageA + (8 * hh + jrow) * kGTN + 4 * (q & 1) + (((j * 4 + 2 * eps + (q >> 1)) ^ sw) << 3);

  f32x16_t acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};

  const ST* live = static_cast<const ST*>(p.live[b]);
  ST* shadow = static_cast<ST*>(p.shadow[b]);
  const float eta = p.eta;

  // fp32 state only: the register epilogue's first live rows are requested
  // with the first stages and held through the main loop (a lane owns 8
  // columns of rows (lane >> 4) + 4 rr of each 16-row step)
  const int c8 = (lane & 15) * 8;
  const int ncol = n0 + c8;
  const bool ncol_ok = ncol < p.d_model;
  Packed<ST, 8> lv[4];
  auto row_of = [&](int sp, int rr) { return m0 + wave * 64 + (sp >> 1) * 32 + (sp & 1) * 16 + (lane >> 4) + 4 * rr; };
  auto load_live = [&](int sp) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int row = row_of(sp, rr);
      if (row < p.d_ff && ncol_ok)
        load_packed<true>(live + size_t(row) * p.d_model + ncol, lv[rr]);
      else
        lv[rr].zero();
    }
  };

  // bf16 state: wave w's 64 live rows are copied into freed stages as two
  // halves of 32 rows x 128 columns (8 KB each), half 0 during the last
  // stage's MFMAs (into the two stages already consumed), half 1 after it
  uint16_t* reg[2] = {s0, s0};
  auto live_copy = [&](uint16_t* dst, int hf) {
    const int row0 = m0 + wave * 64 + hf * 32;
    const int rows = __builtin_amdgcn_readfirstlane(max(0, min(32, p.d_ff - row0)));   // wave-uniform
    const i32x4_t lr = gemm_rsrc(live + size_t(min(row0, p.d_ff)) * p.d_model, rows * p.d_model * 2);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int r = 4 * t + (lane >> 4);
      const int col = n0 + 8 * ((lane & 15) ^ (r & 15));
      const uint32_t off = col < p.d_model ? uint32_t(r * p.d_model + col) * 2u : 0x80000000u;
      gemm_copy<true>(dst + t * 512, off, lr);
    }
  };

  const int nchunks = (p.chunk + kGKC - 1) / kGKC;
  auto step = [&](uint16_t* cur, uint16_t* nxt, uint16_t* oth, int k) {
    // this wave's copies of chunk k are done once at most those of chunk
    // k + 1 are outstanding; the barrier then covers every wave's copies and
    // frees the stage read in step k - 1 for chunk k + 2
    if (k + 1 < nchunks) gemm_wait_vm<kGCopies>();
    else gemm_wait_vm<0>();
    gemm_barrier();
    if (k + 2 < nchunks) issue(nxt, (k + 2) * kGKC);
    if constexpr (sizeof(ST) == 2) {
      if (k + 1 == nchunks) {
        // nxt and oth were read in the two previous steps: 6 free 8 KB slots
        reg[0] = (wave < 2 ? nxt : oth) + (wave & 1) * 4096;
        reg[1] = wave < 3 ? cur + wave * 4096 : nxt + 2 * 4096;
        live_copy(reg[0], 0);
      }
    }
#pragma unroll
    for (int ks = 0; ks < kGKC / 16; ++ks) {
      bf16x8_t af[2], bf[4];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = gemm_operand<kGTM>(cur, offa[i] + ks * 16 * kGTM);
#pragma unroll
      for (int j = 0; j < 4; ++j) bf[j] = gemm_operand<kGTN>(cur, offb[j] + ks * 16 * kGTN);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bf[j], af[i], acc[i][j], 0, 0, 0);
    }
  };

  issue(s0, 0);
  if (nchunks > 1) issue(s1, kGKC);
  if constexpr (sizeof(ST) == 4) load_live(0);
  for (int k = 0; k < nchunks; k += 3) {
    step(s0, s2, s1, k);
    if (k + 1 < nchunks) step(s1, s0, s2, k + 1);
    if (k + 2 < nchunks) step(s2, s1, s0, k + 2);
  }
  // every wave is done with the stages after this barrier
  __builtin_amdgcn_s_waitcnt(0xC07F);                      // lgkmcnt(0)
  gemm_barrier();

  if constexpr (sizeof(ST) == 2) {
    // bf16 state.  The MFMA is issued as D^T = G^T Z, so accumulator register
    // 4a+e of block (i, j) holds D[i*32 + l%32][j*32 + 8a + 4(l/32) + e]:
    // four consecutive columns of one row, the layout of the state itself.
    // Each lane reads those 8 bytes of live from the copied half (row r's
    // 16-byte groups sit in slot (group ^ (r & 15)), so the 16 rows of a
    // half-wave hit distinct banks), forms live + eta * D and writes the
    // bf16 result back in place; whole rows are then read back and stored.
    // Loads and stores go through buffer descriptors clipped to the matrix,
    // so ragged tiles need no branches and every wave issues a fixed number
    // of memory instructions.
    live_copy(reg[1], 1);
    const int ml = lane & 31;                              // row of the half this lane updates
    const int h4 = (lane >> 5) * 4;                        // column offset within the 8-column group
    // store side: lane l moves 16 bytes (8 columns) of row 4t + l / 16, so
    // consecutive lanes write consecutive addresses
    const int srow = lane >> 4;
    const int scol = n0 + 8 * (lane & 15);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      // half 0's copies are done once at most half 1's 8 copies are
      // outstanding (loads complete in order); half 1's were waited for
      // before any store was issued, since stores and loads may complete
      // out of order relative to each other
      if (hf == 0) gemm_wait_vm<8>();
      typedef __attribute__((address_space(3))) u32x2_t lds_u32x2_t;
      u32x2_t lt[4][4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int a = 0; a < 4; ++a)
          lt[j][a] = *(const lds_u32x2_t*)(reg[hf] + ml * kGTN + (((4 * j + a) ^ (ml & 15)) << 3) + h4);
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const f32x16_t& d = acc[hf][j];
          const float f0 = __uint_as_float(lt[j][a][0] << 16) + eta * d[4 * a + 0];
          const float f1 = __uint_as_float(lt[j][a][0] & 0xffff0000u) + eta * d[4 * a + 1];
          const float f2 = __uint_as_float(lt[j][a][1] << 16) + eta * d[4 * a + 2];
          const float f3 = __uint_as_float(lt[j][a][1] & 0xffff0000u) + eta * d[4 * a + 3];
          *(lds_u32x2_t*)(reg[hf] + ml * kGTN + (((4 * j + a) ^ (ml & 15)) << 3) + h4) =
              u32x2_t{bf16x2_rne(f0, f1), bf16x2_rne(f2, f3)};
        }
      asm volatile("" ::: "memory");
      if (hf == 0) gemm_wait_vm<0>();
      const int row0 = m0 + wave * 64 + hf * 32;
      const int rows = __builtin_amdgcn_readfirstlane(max(0, min(32, p.d_ff - row0)));   // wave-uniform
      const __amdgpu_buffer_rsrc_t sr = __builtin_amdgcn_make_buffer_rsrc(
          shadow + size_t(min(row0, p.d_ff)) * p.d_model, (short)0, rows * p.d_model * 2, 0x00020000);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int r = 4 * t + srow;
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(reg[hf] + r * kGTN + (((lane & 15) ^ (r & 15)) << 3));
        const uint32_t off = scol < p.d_model ? uint32_t(r * p.d_model + scol) * 2u : 0x80000000u;
        __builtin_amdgcn_raw_buffer_store_b128(v, sr, off, 0, 2);        // non-temporal
      }
    }
  } else {
    // fp32 state: each wave passes its own accumulators through a private
    // 8 KB LDS region (16 rows x 128 fp32) in 16-row steps, then every lane
    // updates 8 contiguous columns of 4 rows.  Accumulator register 4a+e of
    // block (i, j) holds D[i*32 + l%32][j*32 + 8a + 4(l/32) + e]: the lanes
    // whose row falls in the step write those 16 bytes.  Row r of a region
    // keeps its 16-byte units XOR (r & 15), so the rows of one write hit
    // distinct banks.  LDS requests of one wave complete in order, so the
    // region needs no barrier.
    float* ep = reinterpret_cast<float*>(wave == 1 ? s1 : wave == 2 ? s2 : s0) + (wave == 3 ? 2048 : 0);
    const int hu = lane >> 5;                              // 16-byte unit within the 8-column group
#pragma unroll
    for (int sp = 0; sp < 4; ++sp) {
      const int i = sp >> 1;
      const int qh = sp & 1;
      if (((lane & 31) >> 4) == qh) {
        const int rl = (lane & 15);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int a = 0; a < 4; ++a) {
            const int u = 8 * j + 2 * a + hu;
            *reinterpret_cast<f32x4_t*>(ep + rl * kGTN + ((u ^ rl) << 2)) =
                f32x4_t{acc[i][j][4 * a], acc[i][j][4 * a + 1], acc[i][j][4 * a + 2], acc[i][j][4 * a + 3]};
          }
      }
      asm volatile("" ::: "memory");
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int rl = (lane >> 4) + 4 * rr;
        const int u0 = 2 * (lane & 15);
        const f32x4_t a0 = *reinterpret_cast<const f32x4_t*>(ep + rl * kGTN + ((u0 ^ (rl & 15)) << 2));
        const f32x4_t a1 = *reinterpret_cast<const f32x4_t*>(ep + rl * kGTN + (((u0 + 1) ^ (rl & 15)) << 2));
        const float o[8] = {lv[rr].get(0) + eta * a0[0], lv[rr].get(1) + eta * a0[1],
                            lv[rr].get(2) + eta * a0[2], lv[rr].get(3) + eta * a0[3],
                            lv[rr].get(4) + eta * a1[0], lv[rr].get(5) + eta * a1[1],
                            lv[rr].get(6) + eta * a1[2], lv[rr].get(7) + eta * a1[3]};
        const int row = row_of(sp, rr);
        if (row < p.d_ff && ncol_ok) store_n<8, true>(shadow + size_t(row) * p.d_model + ncol, o);
        // this register slot now takes the same row of the next step
        if (sp + 1 < 4) {
          const int nrow = row_of(sp + 1, rr);
          if (nrow < p.d_ff && ncol_ok)
            load_packed<true>(live + size_t(nrow) * p.d_model + ncol, lv[rr]);
          else
            lv[rr].zero();
        }
      }
      asm volatile("" ::: "memory");
    }
  }
}

// ---------------------------------------------------------------------------
// WRITE, fp32 evidence: VALU rank-C update (fp32 products keep the small
// tiny-config tolerance; bf16 operands would round Z and G)
// ---------------------------------------------------------------------------

template <typename ST>
__global__ void __launch_bounds__(256) write_valu_kernel(const WriteParams p) {
  const int n4 = p.d_model / 4;
  const size_t per_owner = size_t(p.d_ff) * n4;
  const size_t gid = size_t(blockIdx.x) * 256 + threadIdx.x;
  const int b = blockIdx.y;
  if (gid >= per_owner) return;
  const int m = int(gid / n4);
  const int n = int(gid - size_t(m) * n4) * 4;
  const float* Z = static_cast<const float*>(p.z[b]);
  const float* G = static_cast<const float*>(p.g[b]);
  float a[4] = {0.f, 0.f, 0.f, 0.f};
  for (int c = 0; c < p.chunk; ++c) {
    const float zc = Z[size_t(c) * p.d_ff + m];
    const float4 g4 = *reinterpret_cast<const float4*>(G + size_t(c) * p.d_model + n);
    a[0] = fmaf(zc, g4.x, a[0]);
    a[1] = fmaf(zc, g4.y, a[1]);
    a[2] = fmaf(zc, g4.z, a[2]);
    a[3] = fmaf(zc, g4.w, a[3]);
  }
  const ST* live = static_cast<const ST*>(p.live[b]);
  ST* shadow = static_cast<ST*>(p.shadow[b]);
  float lv[4];
  load_n<4>(live + size_t(m) * p.d_model + n, lv);
  float out[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = lv[i] + p.eta * a[i];
  store_n<4, true>(shadow + size_t(m) * p.d_model + n, out);
}

// ---------------------------------------------------------------------------
// TailBufferUpdate for a WRITE step: its own x row becomes the chunk's last
// ---------------------------------------------------------------------------

struct TailParams {
  int n16;                         // 16-byte units per row
  const uint4* x;                  // owner-indexed rows of n16 units
  uint4* dst[RWTTT_MAX_GROUP];
  uint32_t row[RWTTT_MAX_GROUP];
};

__global__ void __launch_bounds__(256) tail_append_kernel(const TailParams p) {
  const int b = blockIdx.y;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < p.n16) p.dst[b][i] = p.x[size_t(p.row[b]) * p.n16 + i];
}

// ---------------------------------------------------------------------------
// Fork: bulk copy of slots and tails (streaming, non-temporal both ways)
// ---------------------------------------------------------------------------

constexpr int kCopyJobs = 64;

struct CopyParams {
  const u32x4_t* src[kCopyJobs];
  u32x4_t* dst[kCopyJobs];
  size_t n16[kCopyJobs];
};

__global__ void __launch_bounds__(256) copy_kernel(const CopyParams p) {
  const int j = blockIdx.y;
  const size_t n = p.n16[j];
  const u32x4_t* s = p.src[j];
  u32x4_t* d = p.dst[j];
  const size_t stride = size_t(gridDim.x) * 256 * 4;
  for (size_t i = size_t(blockIdx.x) * 256 * 4 + threadIdx.x; i < n; i += stride) {
    u32x4_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (i + size_t(u) * 256 < n) v[u] = __builtin_nontemporal_load(s + i + size_t(u) * 256);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (i + size_t(u) * 256 < n) __builtin_nontemporal_store(v[u], d + i + size_t(u) * 256);
  }
}

template <typename IO, typename ST>
hipError_t launch_read_t(const ReadLaunch& L, hipStream_t stream, float* slot_part = nullptr) {
  const ReadGeometry g = read_geometry(L.d_ff, L.d_model, L.state_bf16, L.n_owners);
  ReadParams p;
  p.x = L.x;
  p.y = L.y;
  p.w0 = L.w0;
  p.part = slot_part ? slot_part : static_cast<float*>(L.workspace);
  p.slot_part = slot_part ? 1 : 0;
  p.count = L.count;
  p.d_ff = L.d_ff;
  p.d_model = L.d_model;
  p.ks = g.ks;
  p.nt = g.nt;
  p.npad = g.npad;
  for (int b = 0; b < RWTTT_MAX_GROUP; ++b) {
    p.dw[b] = b < L.count ? L.dw[b] : nullptr;
    p.row[b] = b < L.count ? L.row[b] : 0u;
    p.tail[b] = b < L.count ? L.tail[b] : nullptr;
  }
  // (chunk, tile) pairs rounded up to a multiple of the 8 XCDs
  const unsigned pairs8 = unsigned((g.ks * g.nt + 7) / 8 * 8);
  hipLaunchKernelGGL((read_partial_kernel<IO, ST>), dim3(pairs8 * unsigned(L.count)),
                     dim3(kReadThreads), 0, stream, p);
  hipLaunchKernelGGL((read_reduce_kernel<IO>), dim3((L.d_model + kRedCols - 1) / kRedCols, L.count), dim3(256),
                     0, stream, p);
  return hipGetLastError();
}

template <typename ST>
hipError_t launch_write_t(const WriteLaunch& L, hipStream_t stream) {
  WriteParams p;
  p.count = L.count;
  p.chunk = L.chunk;
  p.d_ff = L.d_ff;
  p.d_model = L.d_model;
  p.eta = L.eta;
  p.parts = 0;
  p.npadw = 0;
  p.x = L.x;
  p.w0 = L.w0;
  p.tpart = nullptr;
  for (int b = 0; b < RWTTT_MAX_GROUP; ++b) {
    const bool in = b < L.count;
    p.live[b] = in ? L.live[b] : nullptr;
    p.shadow[b] = in ? L.shadow[b] : nullptr;
    p.z[b] = in ? L.z[b] : nullptr;
    p.g[b] = in ? L.g[b] : nullptr;
    p.row[b] = in ? L.row[b] : 0u;
  }
  const bool token = L.x != nullptr;
  if (L.io_bf16 && L.chunk <= kSMaxC) {
    const ReadGeometry geo = read_geometry(L.d_ff, L.d_model, L.state_bf16, L.n_owners);
    p.mt = (L.d_ff + kSTM - 1) / kSTM;
    p.ntl = (L.d_model + kSTN - 1) / kSTN;
    // partitions of an owner's row tiles: fixed by the shape, never by the group
    p.parts = std::min(stream_parts(L.d_ff, L.d_model), geo.tparts);
    p.npadw = geo.tnpad;
    p.tpart = token ? reinterpret_cast<float*>(static_cast<char*>(L.workspace) + geo.token_offset) : nullptr;
    const unsigned pairs8 = unsigned((p.ntl * p.parts + 7) / 8 * 8);
    const dim3 grid(pairs8 * unsigned(L.count));
    if (token) {
      hipLaunchKernelGGL((write_stream_kernel<ST, true>), grid, dim3(256), 0, stream, p);
      ReadParams q;
      q.x = nullptr;
      q.y = L.y;
      q.w0 = nullptr;
      q.part = p.tpart;
      q.slot_part = 0;
      q.count = L.count;
      q.d_ff = L.d_ff;
      q.d_model = L.d_model;
      q.ks = p.parts;
      q.nt = p.ntl;
      q.npad = p.npadw;
      for (int b = 0; b < RWTTT_MAX_GROUP; ++b) {
        q.dw[b] = nullptr;
        q.row[b] = b < L.count ? L.row[b] : 0u;
        q.tail[b] = nullptr;
      }
      hipLaunchKernelGGL((read_reduce_kernel<uint16_t>), dim3((L.d_model + kRedCols - 1) / kRedCols, L.count),
                         dim3(256), 0, stream, q);
    } else {
      hipLaunchKernelGGL((write_stream_kernel<ST, false>), grid, dim3(256), 0, stream, p);
    }
    return hipGetLastError();
  }
  if (token) {
    // no fused kernel on this path: the token is an ordinary READ of the group at version v
    ReadLaunch R;
    R.io_bf16 = L.io_bf16;
    R.state_bf16 = L.state_bf16;
    R.d_ff = L.d_ff;
    R.d_model = L.d_model;
    R.count = L.count;
    R.n_owners = L.n_owners;
    R.x = L.x;
    R.y = L.y;
    R.w0 = L.w0;
    R.workspace = L.workspace;
    for (int b = 0; b < L.count; ++b) {
      R.dw[b] = L.live[b];
      R.row[b] = L.row[b];
      R.tail[b] = nullptr;
    }
    const hipError_t e = L.io_bf16 ? launch_read_t<uint16_t, ST>(R, stream)
                                   : launch_read_t<float, ST>(R, stream);
    if (e != hipSuccess) return e;
  }
  if (L.io_bf16) {
    p.mt = (L.d_ff + kGTM - 1) / kGTM;
    p.ntl = (L.d_model + kGTN - 1) / kGTN;
    const unsigned ntg = unsigned((p.ntl + kGColGroups - 1) / kGColGroups);
    const unsigned mtq = unsigned((p.mt + kGRowClasses - 1) / kGRowClasses);
    hipLaunchKernelGGL((write_gemm_kernel<ST>), dim3(unsigned(L.count) * mtq * ntg * 8u), dim3(kGThreads), 0,
                       stream, p);
  } else {
    const size_t per_owner = size_t(L.d_ff) * (L.d_model / 4);
    const unsigned bx = unsigned((per_owner + 255) / 256);
    hipLaunchKernelGGL((write_valu_kernel<ST>), dim3(bx, L.count), dim3(256), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace

ReadGeometry read_geometry(int d_ff, int d_model, int state_bf16, int n_owners) {
  ReadGeometry g;
  const int tile = read_tile_n(state_bf16);
  g.ks = (d_ff + kReadChunk - 1) / kReadChunk;
  g.nt = (d_model + tile - 1) / tile;
  g.npad = g.nt * tile;
  g.part_floats = size_t(n_owners) * g.ks * g.npad;
  // the fused WRITE token's partials follow, also one region per owner
  g.tparts = kSParts;
  g.tnpad = (d_model + kSTN - 1) / kSTN * kSTN;
  g.token_offset = (g.part_floats * sizeof(float) + 255) / 256 * 256;
  g.token_floats = size_t(n_owners) * g.tparts * g.tnpad;
  g.total_bytes = g.token_offset + (g.token_floats * sizeof(float) + 255) / 256 * 256;
  return g;
}

hipError_t launch_read(const ReadLaunch& L, hipStream_t stream) {
  if (L.io_bf16) {
    return L.state_bf16 ? launch_read_t<uint16_t, uint16_t>(L, stream)
                        : launch_read_t<uint16_t, float>(L, stream);
  }
  return L.state_bf16 ? launch_read_t<float, uint16_t>(L, stream)
                      : launch_read_t<float, float>(L, stream);
}

// ---------------------------------------------------------------------------
// READ for callers that cannot allocate device memory
// ---------------------------------------------------------------------------
//
// The split-K partial sums go to a static device array instead of the
// context's workspace, one region per group slot.  Every GPU the library runs
// on holds its own copy of the array until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is only a stand-in): its
// device address is looked up once per device, with that device current, and
// kept.  Every block writes its whole partial tile before the reduce reads it,
// so the array needs no clearing between calls; calls that overlap on one GPU
// share it and race.

static __device__ __align__(256) float scratch[RWTTT_NOALLOC_SCRATCH_BYTES / sizeof(float)];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};   // the array's device address, per device

// The device address of `scratch` on the current device, looked up on the
// first call with that device current.
static hipError_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

size_t read_noalloc_bytes(int d_ff, int d_model, int state_bf16, int count) {
  const ReadGeometry g = read_geometry(d_ff, d_model, state_bf16, count);
  return g.part_floats * sizeof(float);
}

hipError_t launch_read_noalloc(const ReadLaunch& L, hipStream_t stream) {
  if (read_noalloc_bytes(L.d_ff, L.d_model, L.state_bf16, L.count) > RWTTT_NOALLOC_SCRATCH_BYTES)
    return hipErrorInvalidValue;
  void* ptr = nullptr;
  const hipError_t e = scratch_address(&ptr);
  if (e != hipSuccess) return e;
  float* part = static_cast<float*>(ptr);
  if (L.io_bf16) {
    return L.state_bf16 ? launch_read_t<uint16_t, uint16_t>(L, stream, part)
                        : launch_read_t<uint16_t, float>(L, stream, part);
  }
  return L.state_bf16 ? launch_read_t<float, uint16_t>(L, stream, part)
                      : launch_read_t<float, float>(L, stream, part);
}

hipError_t launch_tail_append(const TailLaunch& L, hipStream_t stream) {
  TailParams p;
  p.n16 = L.d_ff * (L.io_bf16 ? 2 : 4) / 16;
  p.x = static_cast<const uint4*>(L.x);
  for (int b = 0; b < RWTTT_MAX_GROUP; ++b) {
    p.dst[b] = b < L.count ? static_cast<uint4*>(L.dst[b]) : nullptr;
    p.row[b] = b < L.count ? L.row[b] : 0u;
  }
  hipLaunchKernelGGL(tail_append_kernel, dim3((p.n16 + 255) / 256, L.count), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_copy(const CopyJob* jobs, int n, hipStream_t stream) {
  for (int first = 0; first < n; first += kCopyJobs) {
    const int m = std::min(kCopyJobs, n - first);
    CopyParams p;
    size_t most = 0;
    for (int j = 0; j < kCopyJobs; ++j) {
      const bool in = j < m;
      p.src[j] = in ? static_cast<const u32x4_t*>(jobs[first + j].src) : nullptr;
      p.dst[j] = in ? static_cast<u32x4_t*>(jobs[first + j].dst) : nullptr;
      p.n16[j] = in ? jobs[first + j].bytes / 16 : 0;
      most = std::max(most, p.n16[j]);
    }
    if (most == 0) continue;
    const size_t blocks = std::min<size_t>((most + 1023) / 1024, 2048);
    hipLaunchKernelGGL(copy_kernel, dim3(unsigned(blocks), unsigned(m)), dim3(256), 0, stream, p);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_write(const WriteLaunch& L, hipStream_t stream) {
  return L.state_bf16 ? launch_write_t<uint16_t>(L, stream) : launch_write_t<float>(L, stream);
}

}  // namespace rwttt
