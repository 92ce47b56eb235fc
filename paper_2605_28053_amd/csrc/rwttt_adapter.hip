// gfx950 kernels of the DeltaAdapterState backend (Section 4.4, backend
// instantiations; Appendix D, the LoRA-style adapter path): each owner's
// request state is a rank-r pair A [d_ff, r], B [r, d_model].
//
// READ  y_r = x_r W0 + (x_r A_r) B_r
// WRITE A' = A + eta Z^T (G B^T),  B' = B + eta (Z A)^T G   (both from the live A, B)
//
// The shared W0 term dominates the READ's bytes; the rank-r terms are tiny.
// Every summation order depends only on the shapes, so an owner's results
// are bit-identical whatever group it is batched in.

#include <algorithm>

#include "rwttt_kernels.h"

namespace rwttt {
namespace {

#include "rwttt_device.h"

constexpr int kAThreads = 1024;   // READ partial blocks: 16 waves share one chunk of rows
constexpr int kAWaves = kAThreads / 64;
constexpr int kAChunk = 192;      // K rows per READ work item
constexpr int kAUnroll = 4;
constexpr int kAGroup = 8;        // owners per READ block: W0 is read once for all of them
constexpr int kARedCols = 64;     // READ reduce: columns per block (four waves split the chunks)
constexpr int kAPQRows = 64;      // evidence rows of P or Q staged per pass of the update

// ---------------------------------------------------------------------------
// READ
// ---------------------------------------------------------------------------
//
// 1. adapter_read_partial_kernel: one 1024-thread block per (K chunk of 256
//    rows, column tile, group of up to 8 owners); each lane streams 16 bytes
//    of every W0 row of the tile once and applies it to all the block's
//    owners, the sixteen waves split the chunk's rows (16 each: four rounds of
//    four loads per wave), and each owner's wave sums
//    are added in wave order into one partial per (owner, chunk, tile).  Owner groups of
//    one (chunk, tile) sit on one XCD (dispatch is round-robin over the 8
//    XCDs).  The chunk's tile blocks also form the owners' chunk shares of
//    u = x A (r values each, ordered two-level sums), owner g in tile
//    g mod (tiles), and the first tile's block appends the x chunk to the
//    owners' tails if asked.
// 2. adapter_read_reduce_kernel: u = sum of the chunks' shares in chunk
//    order; y[n] = (sum of the W0 partials: four contiguous quarters of the
//    chunks, each in chunk order, then the quarters in order) +
//    sum_j u[j] B[j][n], rounded once to the io dtype.

struct AReadParams {
  const void* x;
  void* y;
  const void* w0;
  float* part;        // [n_owners][ks][npad]
  float* upart;       // [n_owners][ks][rank]
  int count, d_ff, d_model, rank, ks, nt, npad;
  const void* state[RWTTT_MAX_GROUP];
  uint32_t row[RWTTT_MAX_GROUP];
  void* tail[RWTTT_MAX_GROUP];
};

template <typename IO, typename ST>
__global__ void __launch_bounds__(kAThreads) adapter_read_partial_kernel(const AReadParams p) {
  constexpr int COLS = 16 / sizeof(IO);
  constexpr int TILE_N = 64 * COLS;
  constexpr int RW = kAChunk / kAWaves;
  __shared__ float xs[kAGroup][kAChunk];
  __shared__ float red[4][kAWaves][TILE_N];
  __shared__ float ured[kAChunk * 8];
  __shared__ float useg[(kAChunk / 8) * 8];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  // block -> (XCD, position) -> ((chunk, tile) pair, owner group)
  const int ngroups = (p.count + kAGroup - 1) / kAGroup;
  const int xcd = blockIdx.x & 7;
  const int pos = blockIdx.x >> 3;
  const int pl = pos / ngroups;
  const int gi = pos - pl * ngroups;
  const int pair = pl * 8 + xcd;
  if (pair >= p.ks * p.nt) return;
  const int kc = pair / p.nt;
  const int nt = pair - kc * p.nt;
  const int k0 = kc * kAChunk;
  const int kn = min(kAChunk, p.d_ff - k0);
  const int col = nt * TILE_N + lane * COLS;
  const bool col_ok = col < p.d_model;
  const int b0 = gi * kAGroup;
  const int ng = min(kAGroup, p.count - b0);

  // this wave's first round of W0 rows is requested before the x staging
  const int kw0 = wave * RW;
  const int kw1 = min(kw0 + RW, kn);
  const IO* wbase = static_cast<const IO*>(p.w0) + size_t(k0) * p.d_model + col;
  Packed<IO, COLS> w[kAUnroll];
#pragma unroll
  for (int u = 0; u < kAUnroll; ++u) {
    if (col_ok && kw0 + u < kw1) load_packed<false>(wbase + size_t(kw0 + u) * p.d_model, w[u]);
    else w[u].zero();
  }

  for (int idx = tid; idx < kAGroup * kAChunk; idx += kAThreads) {
    const int g = idx / kAChunk, k = idx - g * kAChunk;
    xs[g][k] = (g < ng && k < kn)
                   ? Elem<IO>::get(p.x, size_t(p.row[b0 + g]) * p.d_ff + k0 + k) : 0.f;
  }
  if (nt == 0) {
    for (int g = 0; g < ng; ++g) {
      if (p.tail[b0 + g] == nullptr) continue;
      const IO* xr = static_cast<const IO*>(p.x) + size_t(p.row[b0 + g]) * p.d_ff + k0;
      IO* tr = static_cast<IO*>(p.tail[b0 + g]) + k0;
      for (int k = tid; k < kn; k += kAThreads) tr[k] = xr[k];
    }
  }
  __syncthreads();

  // x W0 over this wave's rows for every owner of the group: W0 is read once
  float acc[kAGroup][COLS];
#pragma unroll
  for (int g = 0; g < kAGroup; ++g)
#pragma unroll
    for (int c = 0; c < COLS; ++c) acc[g][c] = 0.f;
  if (col_ok) {
    for (int k = kw0; k < kw1; k += kAUnroll) {
      if (k != kw0) {
#pragma unroll
        for (int u = 0; u < kAUnroll; ++u) {
          if (k + u < kw1) load_packed<false>(wbase + size_t(k + u) * p.d_model, w[u]);
          else w[u].zero();
        }
      }
#pragma unroll
      for (int u = 0; u < kAUnroll; ++u) {
#pragma unroll
        for (int g = 0; g < kAGroup; ++g) {
          const float xv = xs[g][k + u];
#pragma unroll
          for (int c = 0; c < COLS; ++c) acc[g][c] = fmaf(xv, w[u].get(c), acc[g][c]);
        }
      }
    }
  }
  // per owner: the waves' sums in wave order -> one partial per (owner, chunk,
  // tile); four owners per pass through LDS
#pragma unroll
  for (int g0 = 0; g0 < kAGroup; g0 += 4) {
    if (g0 < ng) {
#pragma unroll
      for (int gg = 0; gg < 4; ++gg)
#pragma unroll
        for (int c = 0; c < COLS; ++c) red[gg][wave][lane * COLS + c] = acc[g0 + gg][c];
      __syncthreads();
      for (int idx = tid; idx < 4 * TILE_N; idx += kAThreads) {
        const int gg = idx / TILE_N, j = idx - gg * TILE_N;
        if (g0 + gg < ng) {
          float v = red[gg][0][j];
#pragma unroll
          for (int w = 1; w < kAWaves; ++w) v += red[gg][w][j];
          p.part[(size_t(p.row[b0 + g0 + gg]) * p.ks + kc) * p.npad + nt * TILE_N + j] = v;
        }
      }
      __syncthreads();
    }
  }

  // u share of this chunk for each owner: sum_k x[k] A[k][j], eight rank columns
  // per pass; the chunk's column-tile blocks take the owners in turn (the loop
  // bounds are uniform per block, so every barrier is reached by all threads)
  for (int g = nt; g < ng; g += p.nt) {
    const ST* A = static_cast<const ST*>(p.state[b0 + g]);
    float* ur = p.upart + (size_t(p.row[b0 + g]) * p.ks + kc) * p.rank;
    for (int j0 = 0; j0 < p.rank; j0 += 8) {
      const int k = tid;   // one chunk row per thread of the first 256
      if (k < kAChunk) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const bool ok = k < kn && j0 + j < p.rank;
          ured[k * 8 + j] = ok ? xs[g][k] * Elem<ST>::get(A, size_t(k0 + k) * p.rank + j0 + j) : 0.f;
        }
      }
      __syncthreads();
      if (tid < kAChunk) {
        const int j = tid & 7, seg = tid >> 3;   // 32 segments of 8 rows
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) s += ured[(seg * 8 + i) * 8 + j];
        useg[seg * 8 + j] = s;
      }
      __syncthreads();
      if (tid < 8 && j0 + tid < p.rank) {
        float s = 0.f;
        for (int seg = 0; seg < kAChunk / 8; ++seg) s += useg[seg * 8 + tid];
        ur[j0 + tid] = s;
      }
      __syncthreads();
    }
  }
}

template <typename IO, typename ST>
__global__ void __launch_bounds__(256) adapter_read_reduce_kernel(const AReadParams p) {
  __shared__ float us[8][RWTTT_MAX_RANK];
  __shared__ float u[RWTTT_MAX_RANK];
  const int b = blockIdx.y;
  const int n = blockIdx.x * kARedCols + (threadIdx.x & 63);
  const size_t r = p.row[b];
  {
    // u[j] = sum over chunks of the x A shares: eight strided partial sums per
    // rank column, then those eight in order
    const int j = threadIdx.x & 31, q = threadIdx.x >> 5;
    if (j < p.rank) {
      // chunks q, q + 8, q + 16, ... in order; eight loads in flight at a time
      float s = 0.f;
      for (int kc = q; kc < p.ks; kc += 64) {
        float a[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) a[i] = kc + 8 * i < p.ks ? p.upart[(r * p.ks + kc + 8 * i) * p.rank + j] : 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) s += a[i];
      }
      us[q][j] = s;
    }
    __syncthreads();
    if (int(threadIdx.x) < p.rank) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) s += us[i][threadIdx.x];
      u[threadIdx.x] = s;
    }
    __syncthreads();
  }
  // W0 partials: the four waves sum four contiguous quarters of the chunks,
  // each in chunk order, and the quarters are added in order
  __shared__ float qs[4][kARedCols];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int per = (p.ks + 3) / 4;
  const int k0 = wave * per, k1 = min(p.ks, k0 + per);
  float s = 0.f;
  if (n < p.d_model) {
    const float* q = p.part + r * p.ks * p.npad + n;
    for (int kc = k0; kc < k1; kc += 8) {
      float a[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] = kc + i < k1 ? q[size_t(kc + i) * p.npad] : 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) s += a[i];
    }
  }
  qs[wave][lane] = s;
  __syncthreads();
  if (wave != 0 || n >= p.d_model) return;
  const ST* Bm = static_cast<const ST*>(p.state[b]) + size_t(p.d_ff) * p.rank;
  float lr = 0.f;
  for (int j0 = 0; j0 < p.rank; j0 += 8) {
    float bv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) bv[i] = j0 + i < p.rank ? Elem<ST>::get(Bm, size_t(j0 + i) * p.d_model + n) : 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (j0 + i < p.rank) lr = fmaf(u[j0 + i], bv[i], lr);
  }
  Elem<IO>::put(p.y, r * p.d_model + n, (((qs[0][lane] + qs[1][lane]) + qs[2][lane]) + qs[3][lane]) + lr);
}

// ---------------------------------------------------------------------------
// WRITE
// ---------------------------------------------------------------------------
//
// 1. adapter_pq_kernel: one block per (evidence row c, slice of 1024 columns
//    of G / rows of Z) forms that slice's share of P[c][j] = sum_n G[c][n] B[j][n]
//    or Q[c][j] = sum_k Z[c][k] A[k][j] (four elements per thread, then an
//    ordered two-level sum over the block).
// 2. adapter_update_kernel: one block per 64 rows k of A or columns n of B;
//    its four waves take a quarter of the evidence rows each:
//    A'[k][j] = A[k][j] + eta sum_c Z[c][k] P[c][j] and
//    B'[j][n] = B[j][n] + eta sum_c Q[c][j] G[c][n], each quarter's sum in c
//    order, the quarters added in order; P and Q (their slices added in
//    order) are staged in LDS; the result is written to the shadow slot in
//    the state dtype.

constexpr int kASlice = 1024;    // columns of G / rows of Z per P / Q block
constexpr int kAUpdCols = 64;    // A rows or B columns per update block

struct AWriteParams {
  int count, chunk, d_ff, d_model, rank, max_chunk, sp, sq;   // sp, sq: slices of N, K
  float eta;
  float* P;     // [n_owners][max_chunk][sp][rank] slice shares
  float* Q;     // [n_owners][max_chunk][sq][rank]
  const void* live[RWTTT_MAX_GROUP];
  void* shadow[RWTTT_MAX_GROUP];
  const void* z[RWTTT_MAX_GROUP];
  const void* g[RWTTT_MAX_GROUP];
  uint32_t row[RWTTT_MAX_GROUP];
};

template <typename IO, typename ST>
__global__ void __launch_bounds__(256) adapter_pq_kernel(const AWriteParams p) {
  __shared__ float red[256 * 8];
  __shared__ float seg[32 * 8];
  const int b = blockIdx.z;
  const int c = blockIdx.y;
  const int s = blockIdx.x;                // < sp: a P slice; else a Q slice
  const bool is_p = s < p.sp;
  const int i0 = (is_p ? s : s - p.sp) * kASlice;
  const int lim = is_p ? p.d_model : p.d_ff;
  const ST* A = static_cast<const ST*>(p.live[b]);
  const ST* Bm = A + size_t(p.d_ff) * p.rank;
  const IO* E = static_cast<const IO*>(is_p ? p.g[b] : p.z[b]) + size_t(c) * lim;
  const int tid = threadIdx.x;
  float* out = (is_p ? p.P + ((size_t(p.row[b]) * p.max_chunk + c) * p.sp + s) * p.rank
                     : p.Q + ((size_t(p.row[b]) * p.max_chunk + c) * p.sq + (s - p.sp)) * p.rank);
  for (int j0 = 0; j0 < p.rank; j0 += 8) {
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
#pragma unroll
    for (int e = 0; e < kASlice / 256; ++e) {
      const int i = i0 + e * 256 + tid;
      if (i < lim) {
        const float ev = Elem<IO>::get(E, i);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          if (j0 + j < p.rank) {
            const float f = is_p ? Elem<ST>::get(Bm, size_t(j0 + j) * p.d_model + i)
                                 : Elem<ST>::get(A, size_t(i) * p.rank + j0 + j);
            acc[j] = fmaf(ev, f, acc[j]);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) red[tid * 8 + j] = acc[j];
    __syncthreads();
    {
      const int j = tid & 7, sg = tid >> 3;   // 32 segments of 8 threads
      float t = 0.f;
#pragma unroll
      for (int q = 0; q < 8; ++q) t += red[(sg * 8 + q) * 8 + j];
      seg[sg * 8 + j] = t;
    }
    __syncthreads();
    if (tid < 8 && j0 + tid < p.rank) {
      float t = 0.f;
      for (int sg = 0; sg < 32; ++sg) t += seg[sg * 8 + tid];
      out[j0 + tid] = t;
    }
    __syncthreads();
  }
}

template <typename IO, typename ST>
__global__ void __launch_bounds__(256) adapter_update_kernel(const AWriteParams p) {
  __shared__ float pq[kAPQRows * RWTTT_MAX_RANK];
  __shared__ float part[4][kAUpdCols][RWTTT_MAX_RANK + 1];
  const int b = blockIdx.y;
  const int na = (p.d_ff + kAUpdCols - 1) / kAUpdCols;
  const bool is_a = int(blockIdx.x) < na;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = (is_a ? int(blockIdx.x) : int(blockIdx.x) - na) * kAUpdCols + lane;
  const int lim = is_a ? p.d_ff : p.d_model;
  const int ns = is_a ? p.sp : p.sq;        // A uses P (slices of N); B uses Q (slices of K)
  const float* src = (is_a ? p.P : p.Q) + size_t(p.row[b]) * p.max_chunk * ns * p.rank;
  const IO* E = static_cast<const IO*>(is_a ? p.z[b] : p.g[b]);
  const int ld = is_a ? p.d_ff : p.d_model;
  float acc[RWTTT_MAX_RANK];
#pragma unroll
  for (int j = 0; j < RWTTT_MAX_RANK; ++j) acc[j] = 0.f;
  for (int c0 = 0; c0 < p.chunk; c0 += kAPQRows) {
    const int cn = min(kAPQRows, p.chunk - c0);
    __syncthreads();
    // P / Q rows c0 .. c0+cn: their slice shares added in slice order
    for (int t = threadIdx.x; t < cn * p.rank; t += 256) {
      const int cc = t / p.rank, j = t - cc * p.rank;
      const float* q = src + (size_t(c0 + cc) * ns) * p.rank + j;
      float v = 0.f;
      for (int sl = 0; sl < ns; ++sl) v += q[size_t(sl) * p.rank];
      pq[t] = v;
    }
    __syncthreads();
    // this wave's quarter of the rows, in c order
    const int q0 = (cn * wave) / 4, q1 = (cn * (wave + 1)) / 4;
    if (i < lim) {
      for (int c = q0; c < q1; ++c) {
        const float ev = Elem<IO>::get(E, size_t(c0 + c) * ld + i);
#pragma unroll
        for (int j = 0; j < RWTTT_MAX_RANK; ++j)
          if (j < p.rank) acc[j] = fmaf(ev, pq[c * p.rank + j], acc[j]);
      }
    }
  }
  // the four quarters in wave order
#pragma unroll
  for (int j = 0; j < RWTTT_MAX_RANK; ++j)
    if (j < p.rank) part[wave][lane][j] = acc[j];
  __syncthreads();
  if (i >= lim) return;
  const ST* live = static_cast<const ST*>(p.live[b]);
  ST* shadow = static_cast<ST*>(p.shadow[b]);
  const float eta = p.eta;
  for (int j = wave; j < p.rank; j += 4) {
    const float d = ((part[0][lane][j] + part[1][lane][j]) + part[2][lane][j]) + part[3][lane][j];
    const size_t at = is_a ? size_t(i) * p.rank + j
                           : size_t(p.d_ff) * p.rank + size_t(j) * p.d_model + i;
    Elem<ST>::put(shadow, at, Elem<ST>::get(live, at) + eta * d);
  }
}

template <typename IO, typename ST>
hipError_t launch_adapter_read_t(const AdapterReadLaunch& L, hipStream_t stream) {
  const AdapterGeometry g = adapter_geometry(L.d_ff, L.d_model, L.io_bf16, L.rank, L.n_owners);
  AReadParams p;
  p.x = L.x;
  p.y = L.y;
  p.w0 = L.w0;
  p.part = static_cast<float*>(L.workspace);
  p.upart = reinterpret_cast<float*>(static_cast<char*>(L.workspace) + g.u_offset);
  p.count = L.count;
  p.d_ff = L.d_ff;
  p.d_model = L.d_model;
  p.rank = L.rank;
  p.ks = g.ks;
  p.nt = g.nt;
  p.npad = g.npad;
  for (int b = 0; b < RWTTT_MAX_GROUP; ++b) {
    const bool in = b < L.count;
    p.state[b] = in ? L.state[b] : nullptr;
    p.row[b] = in ? L.row[b] : 0u;
    p.tail[b] = in ? L.tail[b] : nullptr;
  }
  const unsigned pairs8 = unsigned((g.ks * g.nt + 7) / 8 * 8);
  const unsigned groups = unsigned((L.count + kAGroup - 1) / kAGroup);
  hipLaunchKernelGGL((adapter_read_partial_kernel<IO, ST>), dim3(pairs8 * groups),
                     dim3(kAThreads), 0, stream, p);
  hipLaunchKernelGGL((adapter_read_reduce_kernel<IO, ST>), dim3((L.d_model + kARedCols - 1) / kARedCols, L.count),
                     dim3(256), 0, stream, p);
  return hipGetLastError();
}

template <typename IO, typename ST>
hipError_t launch_adapter_write_t(const AdapterWriteLaunch& L, hipStream_t stream) {
  const AdapterGeometry g = adapter_geometry(L.d_ff, L.d_model, L.io_bf16, L.rank, L.n_owners);
  AWriteParams p;
  p.count = L.count;
  p.chunk = L.chunk;
  p.d_ff = L.d_ff;
  p.d_model = L.d_model;
  p.rank = L.rank;
  p.max_chunk = RWTTT_ADAPTER_MAX_CHUNK;
  p.sp = (L.d_model + kASlice - 1) / kASlice;
  p.sq = (L.d_ff + kASlice - 1) / kASlice;
  p.eta = L.eta;
  p.P = reinterpret_cast<float*>(static_cast<char*>(L.workspace) + g.pq_offset);
  p.Q = p.P + size_t(L.n_owners) * RWTTT_ADAPTER_MAX_CHUNK * p.sp * L.rank;
  for (int b = 0; b < RWTTT_MAX_GROUP; ++b) {
    const bool in = b < L.count;
    p.live[b] = in ? L.live[b] : nullptr;
    p.shadow[b] = in ? L.shadow[b] : nullptr;
    p.z[b] = in ? L.z[b] : nullptr;
    p.g[b] = in ? L.g[b] : nullptr;
    p.row[b] = in ? L.row[b] : 0u;
  }
  hipLaunchKernelGGL((adapter_pq_kernel<IO, ST>), dim3(p.sp + p.sq, L.chunk, L.count), dim3(256),
                     0, stream, p);
  const unsigned blocks = unsigned((L.d_ff + kAUpdCols - 1) / kAUpdCols +
                                   (L.d_model + kAUpdCols - 1) / kAUpdCols);
  hipLaunchKernelGGL((adapter_update_kernel<IO, ST>), dim3(blocks, L.count), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

AdapterGeometry adapter_geometry(int d_ff, int d_model, int io_bf16, int rank, int n_owners) {
  AdapterGeometry g;
  const int tile = 64 * (io_bf16 ? 8 : 4);
  g.ks = (d_ff + kAChunk - 1) / kAChunk;
  g.nt = (d_model + tile - 1) / tile;
  g.npad = g.nt * tile;
  g.part_floats = size_t(n_owners) * g.ks * g.npad;
  auto align = [](size_t bytes) { return (bytes + 255) / 256 * 256; };
  g.u_offset = align(g.part_floats * sizeof(float));
  const size_t u_floats = size_t(n_owners) * g.ks * rank;
  g.pq_offset = g.u_offset + align(u_floats * sizeof(float));
  const int slices = (d_model + kASlice - 1) / kASlice + (d_ff + kASlice - 1) / kASlice;
  const size_t pq_floats = size_t(n_owners) * RWTTT_ADAPTER_MAX_CHUNK * slices * rank;
  g.total_bytes = g.pq_offset + align(pq_floats * sizeof(float));
  return g;
}

hipError_t launch_adapter_read(const AdapterReadLaunch& L, hipStream_t stream) {
  if (L.io_bf16) {
    return L.state_bf16 ? launch_adapter_read_t<uint16_t, uint16_t>(L, stream)
                        : launch_adapter_read_t<uint16_t, float>(L, stream);
  }
  return L.state_bf16 ? launch_adapter_read_t<float, uint16_t>(L, stream)
                      : launch_adapter_read_t<float, float>(L, stream);
}

hipError_t launch_adapter_write(const AdapterWriteLaunch& L, hipStream_t stream) {
  if (L.io_bf16) {
    return L.state_bf16 ? launch_adapter_write_t<uint16_t, uint16_t>(L, stream)
                        : launch_adapter_write_t<uint16_t, float>(L, stream);
  }
  return L.state_bf16 ? launch_adapter_write_t<float, uint16_t>(L, stream)
                      : launch_adapter_write_t<float, float>(L, stream);
}

}  // namespace rwttt
