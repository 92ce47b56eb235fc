// Internal launch interface between the host library (rwttt_api.cpp) and the
// gfx950 kernels (rwttt_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "rwttt.h"

namespace rwttt {

// READ tiling.  A work item is (group slot, K chunk, column tile).  The chunk
// and tile sizes depend only on the matrix shape, never on the group, so an
// owner's result does not depend on who else is in the group.
constexpr int kReadThreads = 256;     // 4 wave64s
constexpr int kReadChunk = 256;       // K rows per work item

inline int read_cols_per_lane(int state_bf16) { return state_bf16 ? 8 : 4; }   // 16 B per lane
inline int read_tile_n(int state_bf16) { return 64 * read_cols_per_lane(state_bf16); }

struct ReadGeometry {
  int ks;       // K chunks
  int nt;       // column tiles
  int npad;     // nt * tile_n
  size_t part_floats;    // READ partial sums: n_owners * ks * npad
  int tparts;            // fused WRITE token: row-tile partitions per owner
  int tnpad;             // fused WRITE token: partial row pitch
  size_t token_offset;   // byte offset of the token partials, 256-B aligned
  size_t token_floats;   // n_owners * tparts * tnpad
  size_t total_bytes;    // workspace bytes, 256-B aligned
};

ReadGeometry read_geometry(int d_ff, int d_model, int state_bf16, int n_owners);

struct ReadLaunch {
  int io_bf16, state_bf16;
  int d_ff, d_model, count, n_owners;
  const void* x;             // [n_owners, d_ff], owner-indexed
  void* y;                   // [n_owners, d_model], owner-indexed
  const void* w0;            // [d_ff, d_model]
  void* workspace;           // ReadGeometry layout
  const void* dw[RWTTT_MAX_GROUP];   // live slot of each group slot
  uint32_t row[RWTTT_MAX_GROUP];     // owner id of each group slot
  void* tail[RWTTT_MAX_GROUP];       // tail row that receives the slot's x row, or null
};

// Copy each group slot's x row (owner-indexed, d_ff io elements) to dst[b].
struct TailLaunch {
  int io_bf16, d_ff, count;
  const void* x;
  void* dst[RWTTT_MAX_GROUP];
  uint32_t row[RWTTT_MAX_GROUP];
};

struct WriteLaunch {
  int io_bf16, state_bf16;
  int d_ff, d_model, count, chunk, n_owners;
  float eta;
  const void* x;             // token inputs [n_owners, d_ff], or null for no token
  void* y;                   // token outputs [n_owners, d_model]
  const void* w0;            // W0 of the layer (token only)
  void* workspace;           // ReadGeometry layout (token only)
  const void* live[RWTTT_MAX_GROUP];
  void* shadow[RWTTT_MAX_GROUP];
  const void* z[RWTTT_MAX_GROUP];    // [chunk, d_ff]
  const void* g[RWTTT_MAX_GROUP];    // [chunk, d_model]
  uint32_t row[RWTTT_MAX_GROUP];     // owner id of each group slot
};

hipError_t launch_read(const ReadLaunch& L, hipStream_t stream);

// The same READ with its partial sums in the library's static device array
// (one region per group slot; L.workspace and L.n_owners are not used for
// them).  Allocates nothing.  read_noalloc_bytes() is the array space a call
// needs; a call above RWTTT_NOALLOC_SCRATCH_BYTES returns hipErrorInvalidValue.
size_t read_noalloc_bytes(int d_ff, int d_model, int state_bf16, int count);
hipError_t launch_read_noalloc(const ReadLaunch& L, hipStream_t stream);
hipError_t launch_tail_append(const TailLaunch& L, hipStream_t stream);

// ---- DeltaAdapterState backend (rwttt_adapter.hip) ----
//
// A slot holds A [d_ff, rank] then B [rank, d_model], row-major, state dtype.
// The workspace follows the fast-weight layout (its READ partial region is
// reused for the W0 partial sums, tiled by the io dtype) with the x A partial
// sums and the WRITE's P = G B^T and Q = Z A behind it.
struct AdapterGeometry {
  int ks, nt, npad;          // W0 partial sums: K chunks, column tiles, padded row
  size_t part_floats;        // n_owners * ks * npad
  size_t u_offset;           // bytes: x A partials, n_owners * ks * rank floats
  size_t pq_offset;          // bytes: P then Q, each n_owners * max_chunk * rank floats
  size_t total_bytes;
};
AdapterGeometry adapter_geometry(int d_ff, int d_model, int io_bf16, int rank, int n_owners);

struct AdapterReadLaunch {
  int io_bf16, state_bf16, d_ff, d_model, rank, count, n_owners;
  const void* x;
  void* y;
  const void* w0;
  void* workspace;
  const void* state[RWTTT_MAX_GROUP];   // live slot of each group slot
  uint32_t row[RWTTT_MAX_GROUP];
  void* tail[RWTTT_MAX_GROUP];          // tail row receiving x, or null
};
hipError_t launch_adapter_read(const AdapterReadLaunch& L, hipStream_t stream);

struct AdapterWriteLaunch {
  int io_bf16, state_bf16, d_ff, d_model, rank, count, chunk, n_owners;
  float eta;
  void* workspace;
  const void* live[RWTTT_MAX_GROUP];
  void* shadow[RWTTT_MAX_GROUP];
  const void* z[RWTTT_MAX_GROUP];
  const void* g[RWTTT_MAX_GROUP];
  uint32_t row[RWTTT_MAX_GROUP];
};
hipError_t launch_adapter_write(const AdapterWriteLaunch& L, hipStream_t stream);

// Device-to-device copies of n 16-byte-aligned regions (one launch per 64).
struct CopyJob {
  const void* src;
  void* dst;
  size_t bytes;              // multiple of 16
};
hipError_t launch_copy(const CopyJob* jobs, int n, hipStream_t stream);
hipError_t launch_write(const WriteLaunch& L, hipStream_t stream);

}  // namespace rwttt
