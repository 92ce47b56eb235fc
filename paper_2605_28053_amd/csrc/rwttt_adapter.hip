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
#include <type_traits>

#include "rwttt_kernels.h"

namespace rwttt {
namespace {

#include "rwttt_device.h"

constexpr int kAThreads = 512;    // READ partial blocks: 8 waves, two per SIMD
constexpr int kAWaves = kAThreads / 64;
constexpr int kAChunk = 192;      // K rows per READ work item
constexpr int kARows = kAChunk / kAWaves;   // W0 rows per wave, all requested at once
constexpr int kAGroup = 8;        // owners per READ block: W0 is read once for all of them
constexpr int kAURows = kAChunk / 64;   // chunk rows per lane in the u share
constexpr int kARedCols = 64;     // READ reduce: columns per block (four waves split the chunks)
constexpr int kARedLoads = 16;    // READ reduce: partials in flight per lane
constexpr int kAPQRows = 64;      // evidence rows of P or Q staged per pass of the update

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// x.lo * w.lo + x.hi * w.hi + acc over packed bf16 pairs (v_dot2c_f32_bf16)
__device__ __forceinline__ float dot2_bf16(uint32_t x, uint32_t w, float acc) {
  typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, x), __builtin_bit_cast(bf16x2_v, w),
                                         acc, false);
}

// An empty asm that reads and rewrites four or eight accumulators: the
// arithmetic that produced them cannot move past it.
__device__ __forceinline__ void pin_row(float (&a)[4]) {
  asm volatile("" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]));
}
__device__ __forceinline__ void pin_row(float (&a)[8]) {
  asm volatile("" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(a[4]), "+v"(a[5]),
               "+v"(a[6]), "+v"(a[7]));
}

// Barrier for data exchanged through LDS: this wave's LDS accesses are
// complete, global loads stay in flight (the compiler waits for those where
// their registers are used).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// ---------------------------------------------------------------------------
// READ
// ---------------------------------------------------------------------------
//
// 1. adapter_read_partial_kernel: one 512-thread block per (K chunk of 192
//    rows, column tile, group of up to 8 owners); each lane streams 16 bytes
//    of every W0 row of the tile once and applies it to all the block's
//    owners.  The eight waves split the chunk's rows, 24 each.  A wave requests
//    the x values of its own rows (every owner of the group), then the u
//    share's x and A values, then all of its W0 rows, and only then waits:
//    loads of one wave return in order, so x arrives first, and no wave waits
//    for another's x before requesting W0.  Each owner's wave sums are added
//    in wave order into one partial per (owner, chunk, tile).  Owner groups of
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
__global__ void __launch_bounds__(kAThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
adapter_read_partial_kernel(const AReadParams p) {
  constexpr int COLS = 16 / sizeof(IO);
  constexpr int TILE_N = 64 * COLS;
  __shared__ float xs[kAChunk][kAGroup];   // x chunk, row-major over owners
  // bf16 io: the same chunk as raw bf16, rows 2m and 2m + 1 of an owner in one word
  __shared__ uint16_t xh[sizeof(IO) == 2 ? kAChunk / 2 : 1][kAGroup][2];
  __shared__ float red[kAGroup][kAWaves][TILE_N];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar indexing
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

  // 1. requests, in the order they are needed, every one unconditional
  //    (indices clamped into the buffers, unused values zeroed afterwards) so
  //    that no load waits inside a branch.
  uint32_t rows[kAGroup];   // owner rows of the group's slots (block-uniform)
#pragma unroll
  for (int g = 0; g < kAGroup; ++g) rows[g] = p.row[b0 + min(g, ng - 1)];
  // this wave's x values: its 24 rows of every owner of the group (lane l
  // holds value l + 64 t: owner (l + 64 t) / 24, row (l + 64 t) % 24)
  constexpr int XW = kAGroup * kARows / 64;
  const int kw0 = wave * kARows;
  IO xw[XW];
#pragma unroll
  for (int t = 0; t < XW; ++t) {
    const int idx = lane + 64 * t;
    const int g = idx / kARows, k = idx - g * kARows;
    uint32_t r = rows[0];
#pragma unroll
    for (int g2 = 1; g2 < kAGroup; ++g2) r = g == g2 ? rows[g2] : r;
    xw[t] = static_cast<const IO*>(p.x)[size_t(r) * p.d_ff + k0 + min(kw0 + k, kn - 1)];
  }
  // u share (step 2): wave i takes owner nt + i * tiles of the group; its lanes
  // hold rows lane, lane + 64, lane + 128 of the chunk: their x values and
  // their first eight A columns
  const int ug = nt + wave * p.nt;
  const ST* uA = static_cast<const ST*>(p.state[b0 + (ug < ng ? ug : 0)]);
  const uint32_t urow = p.row[b0 + (ug < ng ? ug : 0)];
  IO xu[kAURows];
  float apre[kAURows][8];
#pragma unroll
  for (int r = 0; r < kAURows; ++r)
    xu[r] = static_cast<const IO*>(p.x)[size_t(urow) * p.d_ff + k0 + min(lane + 64 * r, kn - 1)];
  if (ug < ng) {
#pragma unroll
    for (int r = 0; r < kAURows; ++r) {
      const size_t at = size_t(k0 + min(lane + 64 * r, kn - 1)) * p.rank;
#pragma unroll
      for (int j = 0; j < 8; ++j) apre[r][j] = Elem<ST>::get(uA, at + min(j, p.rank - 1));
    }
  } else {
#pragma unroll
    for (int r = 0; r < kAURows; ++r)
#pragma unroll
      for (int j = 0; j < 8; ++j) apre[r][j] = 0.f;
  }
  // then this wave's W0 rows; rows past the chunk repeat its last row (their
  // x is zero); lanes past d_model read column 0 and their sums are dropped
  const IO* wbase = static_cast<const IO*>(p.w0) + size_t(k0) * p.d_model + (col_ok ? col : 0);
  Packed<IO, COLS> w[kARows];
#pragma unroll
  for (int u = 0; u < kARows; ++u)
    load_packed<false>(wbase + size_t(min(kw0 + u, kn - 1)) * p.d_model, w[u]);
  __builtin_amdgcn_sched_barrier(0);   // every request is out before x is waited for
  // the wave stages its own rows of x (no other wave reads them before the
  // block barrier below; LDS requests of one wave complete in order)
#pragma unroll
  for (int t = 0; t < XW; ++t) {
    const int idx = lane + 64 * t;
    const int g = idx / kARows, k = kw0 + idx - (idx / kARows) * kARows;
    const bool ok = g < ng && k < kn;
    xs[k][g] = ok ? to_f32(xw[t]) : 0.f;
    if constexpr (sizeof(IO) == 2) xh[k >> 1][g][k & 1] = ok ? xw[t] : uint16_t(0);
  }

  // 2. u share of this chunk for the wave's owner: sum_k x[k] A[k][j], eight
  //    rank columns per pass: each lane sums its rows in order, then a
  //    butterfly over the wave (every lane ends with the same sum).  The first
  //    pass uses the requested columns and runs while the W0 rows are still
  //    arriving; passes for ranks above eight load theirs at the end.
  float* ur = p.upart + (size_t(p.row[b0 + (ug < ng ? ug : 0)]) * p.ks + kc) * p.rank;
  auto u_pass = [&](int j0, bool loaded) {
    float sj[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) sj[j] = 0.f;
#pragma unroll
    for (int r = 0; r < kAURows; ++r) {
      const int k = lane + 64 * r;
      const float xk = k < kn ? to_f32(xu[r]) : 0.f;   // zero past the chunk
      const size_t at = size_t(k0 + min(k, kn - 1)) * p.rank;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float a = loaded ? apre[r][j] : Elem<ST>::get(uA, at + min(j0 + j, p.rank - 1));
        sj[j] = fmaf(xk, j0 + j < p.rank ? a : 0.f, sj[j]);
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
#pragma unroll
      for (int j = 0; j < 8; ++j) sj[j] += __shfl_xor(sj[j], m);
    float v = sj[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) v = lane == j ? sj[j] : v;
    if (lane < 8 && j0 + lane < p.rank) ur[j0 + lane] = v;
  };
  if (ug < ng) u_pass(0, true);

  // 3. x W0 over this wave's rows for every owner of the group, rows in order
  float acc[kAGroup][COLS];
#pragma unroll
  for (int g = 0; g < kAGroup; ++g)
#pragma unroll
    for (int c = 0; c < COLS; ++c) acc[g][c] = 0.f;
  if constexpr (sizeof(IO) == 2) {
    // bf16: rows in pairs, one v_dot2 per (owner, column) adds
    // x[2m] W[2m][c] + x[2m+1] W[2m+1][c]; v_perm pairs the two rows' values
    // of a column in one word
#pragma unroll
    for (int m = 0; m < kARows / 2; ++m) {
      const uint32_t* xq = reinterpret_cast<const uint32_t*>(&xh[(kw0 >> 1) + m][0][0]);
      const uint4 xa = *reinterpret_cast<const uint4*>(xq);
      const uint4 xb = *reinterpret_cast<const uint4*>(xq + 4);
      const uint32_t xpair[kAGroup] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
#pragma unroll
      for (int i = 0; i < COLS / 2; ++i) {
        const uint32_t lo = __builtin_amdgcn_perm(w[2 * m + 1].w[i], w[2 * m].w[i], 0x05040100u);
        const uint32_t hi = __builtin_amdgcn_perm(w[2 * m + 1].w[i], w[2 * m].w[i], 0x07060302u);
#pragma unroll
        for (int g = 0; g < kAGroup; ++g) {
          acc[g][2 * i] = dot2_bf16(xpair[g], lo, acc[g][2 * i]);
          acc[g][2 * i + 1] = dot2_bf16(xpair[g], hi, acc[g][2 * i + 1]);
        }
      }
      // one row pair at a time: its x values and paired W0 die before the next
#pragma unroll
      for (int g = 0; g < kAGroup; ++g) pin_row(acc[g]);
    }
  } else {
#pragma unroll
    for (int u = 0; u < kARows; ++u) {
      float xr[kAGroup];
#pragma unroll
      for (int g = 0; g < kAGroup; g += 4) {
        const float4 x4 = *reinterpret_cast<const float4*>(&xs[kw0 + u][g]);
        xr[g] = x4.x; xr[g + 1] = x4.y; xr[g + 2] = x4.z; xr[g + 3] = x4.w;
      }
#pragma unroll
      for (int g = 0; g < kAGroup; ++g)
#pragma unroll
        for (int c = 0; c < COLS; ++c) acc[g][c] = fmaf(xr[g], w[u].get(c), acc[g][c]);
      // one row at a time: the row's products are done here, so its x values
      // and converted W0 die before the next row's are formed
#pragma unroll
      for (int g = 0; g < kAGroup; ++g) pin_row(acc[g]);
    }
  }

  // 4. per owner: the waves' sums in wave order -> one partial per (owner,
  //    chunk, tile), all owners in one pass through LDS
#pragma unroll
  for (int g = 0; g < kAGroup; ++g)
#pragma unroll
    for (int c = 0; c < COLS; c += 4)
      *reinterpret_cast<float4*>(&red[g][wave][lane * COLS + c]) =
          col_ok ? make_float4(acc[g][c], acc[g][c + 1], acc[g][c + 2], acc[g][c + 3])
                 : make_float4(0.f, 0.f, 0.f, 0.f);
  lds_barrier();
  for (int idx = tid; idx < kAGroup * TILE_N / 4; idx += kAThreads) {
    const int g = idx / (TILE_N / 4), j = (idx - g * (TILE_N / 4)) * 4;
    if (g < ng) {
      float4 v = *reinterpret_cast<const float4*>(&red[g][0][j]);
#pragma unroll
      for (int w2 = 1; w2 < kAWaves; ++w2) {
        const float4 t = *reinterpret_cast<const float4*>(&red[g][w2][j]);
        v.x += t.x; v.y += t.y; v.z += t.z; v.w += t.w;
      }
      uint32_t r = rows[0];
#pragma unroll
      for (int g2 = 1; g2 < kAGroup; ++g2) r = g == g2 ? rows[g2] : r;
      *reinterpret_cast<float4*>(p.part + (size_t(r) * p.ks + kc) * p.npad + nt * TILE_N + j) = v;
    }
  }

  if (ug < ng)
    for (int j0 = 8; j0 < p.rank; j0 += 8) u_pass(j0, false);

  // 5. TailBufferUpdate: the first tile's block appends the staged x chunk
  if (nt == 0) {
    for (int g = 0; g < ng; ++g) {
      if (p.tail[b0 + g] == nullptr) continue;
      for (int k = tid; k < kn; k += kAThreads) Elem<IO>::put(p.tail[b0 + g], k0 + k, xs[k][g]);
    }
  }
}

template <typename IO, typename ST>
__global__ void __launch_bounds__(256) adapter_read_reduce_kernel(const AReadParams p) {
  __shared__ float us[8][RWTTT_MAX_RANK];
  __shared__ float u[RWTTT_MAX_RANK];
  __shared__ float qs[4][kARedCols];
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = blockIdx.x * kARedCols + lane;
  const int nc = min(n, p.d_model - 1);
  const size_t r = p.row[b];
  const int per = (p.ks + 3) / 4;
  const int k0 = wave * per, k1 = min(p.ks, k0 + per);
  const float* q = p.part + r * p.ks * p.npad + nc;
  const int j = threadIdx.x & 31, qq = threadIdx.x >> 5;
  const ST* Bm = static_cast<const ST*>(p.state[b]) + size_t(p.d_ff) * p.rank;

  // 1. every first-round request at once, unconditional (indices clamped,
  //    unused values dropped below): this lane's W0 partials (its wave's
  //    quarter of the chunks), its x A shares (chunks qq, qq + 8, ...) and the
  //    first eight B values of its column
  float a[kARedLoads], t[8], bv[8];
#pragma unroll
  for (int i = 0; i < kARedLoads; ++i) a[i] = q[size_t(min(k0 + i, p.ks - 1)) * p.npad];
#pragma unroll
  for (int i = 0; i < 8; ++i)
    t[i] = p.upart[(r * p.ks + min(qq + 8 * i, p.ks - 1)) * p.rank + min(j, p.rank - 1)];
#pragma unroll
  for (int i = 0; i < 8; ++i) bv[i] = Elem<ST>::get(Bm, size_t(min(i, p.rank - 1)) * p.d_model + nc);

  // 2. W0 partials: the four waves sum four contiguous quarters of the
  //    chunks, each in chunk order, and the quarters are added in order
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kARedLoads; ++i) s += k0 + i < k1 ? a[i] : 0.f;
  for (int kc = k0 + kARedLoads; kc < k1; kc += 8) {
    float a2[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) a2[i] = kc + i < k1 ? q[size_t(kc + i) * p.npad] : 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += a2[i];
  }
  qs[wave][lane] = s;
  // u[j] = sum over chunks of the x A shares: eight strided partial sums per
  // rank column (chunks qq, qq + 8, qq + 16, ... in order), then those eight in order
  if (j < p.rank) {
    float su = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) su += qq + 8 * i < p.ks ? t[i] : 0.f;
    for (int kc = qq + 64; kc < p.ks; kc += 64) {
      float t2[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) t2[i] = kc + 8 * i < p.ks ? p.upart[(r * p.ks + kc + 8 * i) * p.rank + j] : 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) su += t2[i];
    }
    us[qq][j] = su;
  }
  lds_barrier();
  if (int(threadIdx.x) < p.rank) {
    float su = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) su += us[i][threadIdx.x];
    u[threadIdx.x] = su;
  }
  lds_barrier();
  if (wave != 0 || n >= p.d_model) return;
  // 3. + u B, rank columns in order
  float lr = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
    if (i < p.rank) lr = fmaf(u[i], bv[i], lr);
  for (int j0 = 8; j0 < p.rank; j0 += 8) {
    float b2[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) b2[i] = j0 + i < p.rank ? Elem<ST>::get(Bm, size_t(j0 + i) * p.d_model + n) : 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (j0 + i < p.rank) lr = fmaf(u[j0 + i], b2[i], lr);
  }
  Elem<IO>::put(p.y, r * p.d_model + n, (((qs[0][lane] + qs[1][lane]) + qs[2][lane]) + qs[3][lane]) + lr);
}

// ---------------------------------------------------------------------------
// WRITE
// ---------------------------------------------------------------------------
//
// 1. adapter_pq_kernel: one block per (evidence row c, slice of 1024 columns
//    of G / rows of Z) forms that slice's share of P[c][j] = sum_n G[c][n] B[j][n]
//    or Q[c][j] = sum_k Z[c][k] A[k][j] (four elements per thread in order, a
//    butterfly in each wave, then the four waves in order).
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
  constexpr int EPT = kASlice / 256;       // evidence elements per thread
  constexpr int kQLoads = 32;              // A requests in flight per thread (Q, power-of-two rank)
  __shared__ float wsum[4][RWTTT_MAX_RANK];
  __shared__ float zs[kASlice];
  const int b = blockIdx.z;
  const int c = blockIdx.y;
  const int s = blockIdx.x;                // < sp: a P slice; else a Q slice
  const bool is_p = s < p.sp;
  const int i0 = (is_p ? s : s - p.sp) * kASlice;
  const int lim = is_p ? p.d_model : p.d_ff;
  const ST* A = static_cast<const ST*>(p.live[b]);
  const ST* F = is_p ? A + size_t(p.d_ff) * p.rank : A;   // B for P, A for Q
  const IO* E = static_cast<const IO*>(is_p ? p.g[b] : p.z[b]) + size_t(c) * lim;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float* out = (is_p ? p.P + ((size_t(p.row[b]) * p.max_chunk + c) * p.sp + s) * p.rank
                     : p.Q + ((size_t(p.row[b]) * p.max_chunk + c) * p.sq + (s - p.sp)) * p.rank);
  // requests first, unconditional (indices clamped, unused values dropped):
  // the evidence elements, then each rank pass's factor values
  float ev[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) ev[e] = Elem<IO>::get(E, min(i0 + e * 256 + tid, lim - 1));
  const int r = p.rank;
  if (!is_p && (r & (r - 1)) == 0) {
    // Q with a power-of-two rank: the slice's A rows are one contiguous run of
    // 1024 r floats; thread t reads flat elements t, t + 256, ... (consecutive
    // lanes on consecutive addresses), all of rank column t mod r, against
    // the Z values of their rows staged in LDS.  Per thread in flat order,
    // then a butterfly over the lanes of one column, then the waves in order.
#pragma unroll
    for (int e = 0; e < EPT; ++e) zs[e * 256 + tid] = i0 + e * 256 + tid < lim ? ev[e] : 0.f;
    lds_barrier();
    const int lr = __builtin_ctz(r);
    const size_t base = size_t(i0) * r, last = size_t(p.d_ff) * r - 1;
    float acc = 0.f;
    for (int m0 = 0; m0 < 4 * r; m0 += kQLoads) {
      float a[kQLoads];
#pragma unroll
      for (int q = 0; q < kQLoads; ++q)
        a[q] = Elem<ST>::get(A, min(base + size_t(tid + 256 * min(m0 + q, 4 * r - 1)), last));
#pragma unroll
      for (int q = 0; q < kQLoads; ++q)
        if (m0 + q < 4 * r) acc = fmaf(zs[(tid + 256 * (m0 + q)) >> lr], a[q], acc);
    }
    for (int m = 32; m >= r; m >>= 1) acc += __shfl_xor(acc, m);
    if (lane < r) wsum[wave][lane] = acc;
    lds_barrier();
    if (tid < r) out[tid] = ((wsum[0][tid] + wsum[1][tid]) + wsum[2][tid]) + wsum[3][tid];
    return;
  }
  for (int j0 = 0; j0 < p.rank; j0 += 8) {
    float f[EPT][8];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int ic = min(i0 + e * 256 + tid, lim - 1);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int jj = min(j0 + j, p.rank - 1);
        f[e][j] = Elem<ST>::get(F, is_p ? size_t(jj) * p.d_model + ic : size_t(ic) * p.rank + jj);
      }
    }
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const float x = i0 + e * 256 + tid < lim ? ev[e] : 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = fmaf(x, f[e][j], acc[j]);
    }
    // the block's sum: a butterfly in each wave, then the four waves in order
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] += __shfl_xor(acc[j], m);
    if (lane == 0) {
#pragma unroll
      for (int j = 0; j < 8; ++j) wsum[wave][j] = acc[j];
    }
    lds_barrier();
    if (tid < 8 && j0 + tid < p.rank)
      out[j0 + tid] = ((wsum[0][tid] + wsum[1][tid]) + wsum[2][tid]) + wsum[3][tid];
    lds_barrier();
  }
}

template <typename IO, typename ST>
__global__ void __launch_bounds__(256) adapter_update_kernel(const AWriteParams p) {
  constexpr int RPW = kAPQRows / 4;        // evidence rows per wave and pass
  constexpr int kPQItems = 2;              // P / Q items per thread whose shares are requested early
  __shared__ float pq[kAPQRows * RWTTT_MAX_RANK];
  __shared__ float part[4][kAUpdCols][RWTTT_MAX_RANK + 1];
  const int b = blockIdx.y;
  const int na = (p.d_ff + kAUpdCols - 1) / kAUpdCols;
  const bool is_a = int(blockIdx.x) < na;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = (is_a ? int(blockIdx.x) : int(blockIdx.x) - na) * kAUpdCols + lane;
  const int lim = is_a ? p.d_ff : p.d_model;
  const int ic = min(i, lim - 1);
  const int ns = is_a ? p.sp : p.sq;        // A uses P (slices of N); B uses Q (slices of K)
  const float* src = (is_a ? p.P : p.Q) + size_t(p.row[b]) * p.max_chunk * ns * p.rank;
  const IO* E = static_cast<const IO*>(is_a ? p.z[b] : p.g[b]);
  const int ld = is_a ? p.d_ff : p.d_model;
  const ST* live = static_cast<const ST*>(p.live[b]);
  ST* shadow = static_cast<ST*>(p.shadow[b]);
  auto at_of = [&](int j) {
    return is_a ? size_t(ic) * p.rank + j : size_t(p.d_ff) * p.rank + size_t(j) * p.d_model + ic;
  };
  // the live values of the first two rank columns this thread finishes
  // (j = wave, wave + 4), requested first
  float lv[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) lv[h] = Elem<ST>::get(live, at_of(min(wave + 4 * h, p.rank - 1)));
  float acc[RWTTT_MAX_RANK];
#pragma unroll
  for (int j = 0; j < RWTTT_MAX_RANK; ++j) acc[j] = 0.f;
  for (int c0 = 0; c0 < p.chunk; c0 += kAPQRows) {
    const int cn = min(kAPQRows, p.chunk - c0);
    // this wave's quarter of the pass's rows, in c order
    const int q0 = (cn * wave) / 4, q1 = (cn * (wave + 1)) / 4;
    float ev[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) ev[r] = Elem<IO>::get(E, size_t(c0 + min(q0 + r, cn - 1)) * ld + ic);
    // P / Q rows c0 .. c0+cn: their slice shares added in slice order.  The
    // first kPQItems items of each thread have their first NS shares
    // requested at once, before the barrier that frees pq (NS: the slice
    // count rounded up to 4, 8 or 16); further shares are loaded after it.
    const int items = cn * p.rank;
    auto stage = [&](auto nsl) {
      constexpr int NS = decltype(nsl)::value;
      float sh[kPQItems][NS];
#pragma unroll
      for (int it = 0; it < kPQItems; ++it) {
        const int t = min(int(threadIdx.x) + 256 * it, items - 1);
        const int cc = t / p.rank, j = t - cc * p.rank;
        const float* q = src + (size_t(c0 + cc) * ns) * p.rank + j;
#pragma unroll
        for (int sl = 0; sl < NS; ++sl) sh[it][sl] = q[size_t(min(sl, ns - 1)) * p.rank];
      }
      lds_barrier();   // the previous pass's P / Q rows are no longer read
      for (int t = threadIdx.x, it = 0; t < items; t += 256, ++it) {
        const int cc = t / p.rank, j = t - cc * p.rank;
        const float* q = src + (size_t(c0 + cc) * ns) * p.rank + j;
        float v = 0.f;
        if (it < kPQItems) {
#pragma unroll
          for (int sl = 0; sl < NS; ++sl) v += sl < ns ? (it == 0 ? sh[0][sl] : sh[kPQItems - 1][sl]) : 0.f;
        }
        for (int sl0 = it < kPQItems ? NS : 0; sl0 < ns; sl0 += 8) {
          float a2[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) a2[k] = q[size_t(min(sl0 + k, ns - 1)) * p.rank];
#pragma unroll
          for (int k = 0; k < 8; ++k) v += sl0 + k < ns ? a2[k] : 0.f;
        }
        pq[t] = v;
      }
    };
    if (ns <= 4) stage(std::integral_constant<int, 4>{});
    else if (ns <= 8) stage(std::integral_constant<int, 8>{});
    else stage(std::integral_constant<int, 16>{});
    lds_barrier();
    // this wave's rows in c order; the rank loop is branch-free (columns past
    // the rank read a valid pq entry and are never stored)
    auto rows = [&](auto rk) {
      constexpr int R = decltype(rk)::value;
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
        if (q0 + r < q1) {
          const float* row = pq + (q0 + r) * p.rank;
#pragma unroll
          for (int j = 0; j < R; ++j) acc[j] = fmaf(ev[r], row[min(j, p.rank - 1)], acc[j]);
        }
      }
    };
    if (p.rank <= 8) rows(std::integral_constant<int, 8>{});
    else if (p.rank <= 16) rows(std::integral_constant<int, 16>{});
    else rows(std::integral_constant<int, RWTTT_MAX_RANK>{});
  }
  // the four quarters in wave order
#pragma unroll
  for (int j = 0; j < RWTTT_MAX_RANK; ++j)
    if (j < p.rank) part[wave][lane][j] = acc[j];
  lds_barrier();
  if (i >= lim) return;
  const float eta = p.eta;
  for (int j = wave, h = 0; j < p.rank; j += 4, ++h) {
    const float d = ((part[0][lane][j] + part[1][lane][j]) + part[2][lane][j]) + part[3][lane][j];
    const float l = h == 0 ? lv[0] : h == 1 ? lv[1] : Elem<ST>::get(live, at_of(j));
    Elem<ST>::put(shadow, at_of(j), l + eta * d);
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
