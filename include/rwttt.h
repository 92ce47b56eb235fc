/*
 * rwttt.h -- C ABI of the owner-scoped fast-weight READ/WRITE path of
 * read-write TTT serving (RW-TTT, Yang et al.), for AMD Instinct MI355X
 * (gfx950).
 *
 * Every request r owns a versioned state per layer that modifies the shared
 * down-projection W0 (Section 3, request tuple and Ownership; Section 4.1):
 * a fast-weight delta dW_r (FastWeightState) or a low-rank pair A_r, B_r
 * (DeltaAdapterState, Section 4.4).  The library keeps, per (owner, layer),
 * two caller-allocated device slots: the live slot holds the committed
 * version V(r), the other is the shadow that receives a WRITE's dirty
 * candidate.  Commit flips which slot is live; rollback forgets the shadow.
 * Neither copies state.
 *
 * Conventions for every entry point:
 *  - Returns an rwttt_status: RWTTT_OK (0) or a negative error code.
 *  - Arguments are validated before anything changes; on error the owner
 *    table is left as it was and nothing is launched.
 *  - Device pointers are plain HIP device addresses, 16-byte aligned.  The
 *    caller allocates and frees all device memory (weights, slots, inputs,
 *    outputs, workspace); the library never allocates or frees device memory
 *    and never synchronises the stream it is given.
 *  - Host arrays are read during the call only; the library keeps no pointer
 *    to them, except the config's pointer tables, which it copies.
 *  - Matrices are row-major.  Shapes: W0 [d_ff, d_model]; a fast-weight slot
 *    [d_ff, d_model], an adapter slot A [d_ff, r] then B [r, d_model];
 *    x [n_owners, d_ff]; y [n_owners, d_model]; Z [C, d_ff]; G [C, d_model].
 *  - A context is not thread-safe; use one per host thread.
 */
#ifndef RWTTT_H
#define RWTTT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t rwttt_status;

/* status codes */
#define RWTTT_OK               0
#define RWTTT_DEFERRED         1   /* per-event plan status: held back by the wait budget */
#define RWTTT_E_INVALID       -1   /* bad argument, shape, pointer or owner id          */
#define RWTTT_E_STALE_VERSION -2   /* event's expected version differs from V(r)        */
#define RWTTT_E_OWNER_ALIAS   -3   /* one owner appears twice in an event set or group  */
#define RWTTT_E_KEY_MISMATCH  -4   /* wrong effect for the call                         */
#define RWTTT_E_NOT_DIRTY     -5   /* commit/rollback of an owner with no candidate     */
#define RWTTT_E_DIRTY         -6   /* owner already holds an uncommitted candidate      */
#define RWTTT_E_CAPACITY      -7   /* an output array is too small                      */
#define RWTTT_E_HIP           -8   /* HIP launch or runtime error; see rwttt_last_hip_error */
#define RWTTT_E_WRITE_FAILED  -9   /* a WRITE of this owner failed; it can only roll back */

/* state effect rho (Section 3, eq. event) */
#define RWTTT_READ  0
#define RWTTT_WRITE 1

/* element types */
#define RWTTT_F32  0
#define RWTTT_BF16 1   /* bfloat16, round-to-nearest-even on every narrowing */

/* largest owner group one rwttt_read / rwttt_write call accepts */
#define RWTTT_MAX_GROUP 64

/* backend types tau (Section 4.1 payloads; Section 4.4 backend instantiations) */
#define RWTTT_FAST_WEIGHT    0   /* FastWeightState: dW [d_ff, d_model] per (owner, layer)   */
#define RWTTT_DELTA_ADAPTER  1   /* DeltaAdapterState: low-rank A [d_ff, r], B [r, d_model]   */
#define RWTTT_MAX_RANK      32   /* largest adapter rank r                                     */
#define RWTTT_ADAPTER_MAX_CHUNK 1024   /* largest WRITE chunk C of the adapter backend        */

typedef struct rwttt_ctx rwttt_ctx;

/* One ready transition e_i = (r_i, tau_i, sigma_i, rho_i, v_i) plus its ready
 * step (Section 3, eqs. event and wait-budget).  The planner compares
 * backend_type, shape_class and placement only for equality and order. */
typedef struct rwttt_event {
    uint32_t owner;             /* r: owner id, < n_owners                     */
    uint32_t backend_type;      /* tau: backend state type                     */
    uint32_t shape_class;       /* sigma: operator shape class (opaque)        */
    uint32_t placement;         /* pi: placement (device)                      */
    int32_t  effect;            /* rho: RWTTT_READ or RWTTT_WRITE              */
    uint32_t reserved;          /* must be 0                                   */
    uint64_t expected_version;  /* v_i, checked against V(r_i)                 */
    uint64_t ready_step;        /* decode step at which the event became ready */
} rwttt_event;

/* One legal group: all members share kappa = (rho, tau, sigma, pi); its
 * owner map is owner_map[first .. first+count) (Section 4.3). */
typedef struct rwttt_group {
    int32_t  effect;
    uint32_t backend_type;
    uint32_t shape_class;
    uint32_t placement;
    uint32_t first;
    uint32_t count;
} rwttt_group;

typedef struct rwttt_config {
    uint32_t n_owners;          /* number of request owners                       */
    uint32_t n_layers;          /* fast-weight layers per owner                   */
    uint32_t d_ff;              /* rows of W0 and of each slot; multiple of 8     */
    uint32_t d_model;           /* columns; multiple of 8                         */
    int32_t  io_dtype;          /* RWTTT_F32 / RWTTT_BF16: x, W0, y, Z, G         */
    int32_t  state_dtype;       /* RWTTT_F32 / RWTTT_BF16: fast-weight slots      */
    uint32_t max_group;         /* largest group a call accepts, 1..RWTTT_MAX_GROUP */
    uint32_t backend;           /* RWTTT_FAST_WEIGHT or RWTTT_DELTA_ADAPTER       */
    uint32_t rank;              /* adapter rank r, 1..RWTTT_MAX_RANK, for
                                   RWTTT_DELTA_ADAPTER; must be 0 otherwise       */
    uint32_t reserved;          /* must be 0                                      */
    const void* const* w0;      /* [n_layers] device pointers to W0_l             */
    void* const* slots;         /* [n_owners*n_layers*2] device pointers; entry
                                   (owner*n_layers + layer)*2 + s is slot s.
                                   Slot 0 holds version 0 and starts live.
                                   A fast-weight slot is dW [d_ff, d_model]; an
                                   adapter slot is A [d_ff, r] followed by
                                   B [r, d_model] (rwttt_slot_bytes).            */
    void* workspace;            /* device buffer of rwttt_workspace_bytes() bytes,
                                   or NULL for a host-only context (planning and
                                   the owner table): every call that would touch
                                   the device (read, write, fork, checkpoint,
                                   resume) then returns RWTTT_E_INVALID */
    size_t workspace_bytes;
} rwttt_config;

/* Bytes of device workspace a context with this config needs: the READ
 * split-K partial sums, n_owners x ceil(d_ff/256) x d_model fp32 values
 * (d_model rounded up to the column tile), and the fused WRITE token's
 * partial sums, n_owners x 64 x d_model fp32 values (one per row-tile
 * partition of the streaming WRITE; the shape fixes at most 64 of them,
 * d_model rounded up to 256); for the adapter backend
 * also n_owners x ceil(d_ff/256) x r partial sums of x A and two
 * n_owners x RWTTT_ADAPTER_MAX_CHUNK x r scratch matrices of a WRITE; one
 * region per owner.  Only the shape fields are read.  The workspace needs no
 * initialisation. */
rwttt_status rwttt_workspace_bytes(const rwttt_config* cfg, size_t* bytes);

/* Bytes of one state slot: d_ff * d_model (fast weights) or
 * (d_ff + d_model) * r (adapter) elements of the state dtype. */
rwttt_status rwttt_slot_bytes(const rwttt_config* cfg, size_t* bytes);

/* Create a context: copies the pointer tables, sets V(r) = 0, slot 0 live and
 * no candidate for every owner.  Makes no HIP call.  Slot pointers must be
 * pairwise distinct (RWTTT_E_OWNER_ALIAS otherwise).  *out is set only on
 * success; release with rwttt_destroy. */
rwttt_status rwttt_create(const rwttt_config* cfg, rwttt_ctx** out);
rwttt_status rwttt_destroy(rwttt_ctx* ctx);

/* LegalGroups (Algorithm 1; Section 3 eqs. compatibility and wait-budget;
 * Section 4.3).  Host-only, integer-only, reads the owner table and changes
 * nothing.
 *   ev[n_ev]        ready events at decode step `step`.
 *   target_b        target group size B (0: no size target).
 *   wait_budget     w: a partial group is issued only when w == 0 or its
 *                   oldest member has waited w steps; otherwise deferred.
 * Outputs: groups[0 .. *n_groups) in key order (effect, backend_type,
 * shape_class, placement as unsigned integers, READ first), each group's
 * members in (ready_step, owner) order, concatenated in owner_map; deferred
 * event indices in the same order; ev_status[i] = RWTTT_OK (issued),
 * RWTTT_DEFERRED, or a rejection: RWTTT_E_INVALID (bad owner/effect, or
 * ready_step > step), RWTTT_E_DIRTY (owner holds a candidate),
 * RWTTT_E_STALE_VERSION (expected_version != V(owner)).
 * Returns RWTTT_E_OWNER_ALIAS if two events name one owner (then no output is
 * meaningful), RWTTT_E_CAPACITY if groups_cap, map_cap or deferred_cap is too
 * small (*n_groups, *n_mapped and *n_deferred then hold the sizes needed). */
rwttt_status rwttt_plan(const rwttt_ctx* ctx, const rwttt_event* ev, uint32_t n_ev,
                        uint64_t step, uint32_t target_b, uint32_t wait_budget,
                        rwttt_group* groups, uint32_t groups_cap, uint32_t* n_groups,
                        uint32_t* owner_map, uint32_t map_cap, uint32_t* n_mapped,
                        uint32_t* deferred, uint32_t deferred_cap, uint32_t* n_deferred,
                        int32_t* ev_status);

/* READ / ApplyState (Section 3, Read; Section 4.2 primitives table): for each
 * slot b of the group, owner r = owner_map[first+b]:
 *     y[r, :] = x[r, :] W0_layer + x[r, :] dW_{r,layer}^live          (fast weights)
 *     y[r, :] = x[r, :] W0_layer + (x[r, :] A_{r,layer}) B_{r,layer}   (adapter)
 * accumulated in fp32 and rounded once to the io dtype.  Versions and slots
 * are unchanged.  Also emits the token of a WRITE step, read at version v
 * before its candidate is committed (Section 3, Write returns y; Section 4.1,
 * the candidate is invisible until commit), so `group` may have either
 * effect.  x and y are owner-indexed: only the group's rows are read or
 * written, which returns outputs through the owner map (Algorithm 1,
 * ReturnOutputs).  y must not overlap x, W0 or any slot.  Results for an owner
 * are bit-identical whatever the group's size, order or other members.
 * An empty group returns RWTTT_OK and launches nothing.  Launches two kernels
 * on `stream` (split-K partial sums into the owners' workspace regions, then
 * their reduction).  Reads and writes of one context may run concurrently on
 * different streams when they name disjoint owners (the serving contract
 * gives each owner one transition per step); calls that share an owner must
 * be ordered on the device (same stream, or an event wait).
 *
 * expected: NULL, or a host array indexed like owner_map (entry first+b
 * belongs to slot b) holding the version each member was planned at
 * (the event's v_i).  Every member must still be at it (Section 3, eq.
 * compatibility: a group executes only members at their committed version);
 * otherwise the call returns RWTTT_E_STALE_VERSION and launches nothing.
 * The planner already guarantees this for a plan used in the same step;
 * the check catches a group built by hand or kept across a commit. */
rwttt_status rwttt_read(rwttt_ctx* ctx, const rwttt_group* group, const uint32_t* owner_map,
                        const uint64_t* expected, uint32_t layer, const void* x, void* y,
                        void* stream);

/* Largest device scratch rwttt_read_noalloc uses: its static array's size. */
#define RWTTT_NOALLOC_SCRATCH_BYTES (16u << 20)

/* rwttt_read for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  The
 * same computation, kernels and results as rwttt_read (bit for bit), but the
 * split-K partial sums go to a static device array of
 * RWTTT_NOALLOC_SCRATCH_BYTES inside the library instead of the context's
 * workspace, so the context may be a host-only one (workspace NULL).  The
 * call allocates and frees nothing.  A group needs
 * count x ceil(d_ff/256) x d_model fp32 values of the array (d_model rounded
 * up to the column tile: 256 for fp32 state, 512 for bf16 state); a larger
 * group returns RWTTT_E_CAPACITY.  Fast-weight backend only (RWTTT_E_INVALID
 * for an adapter context); no tail append.  The stream must belong to the
 * current device: each GPU holds its own copy of the array (until the process
 * ends), found on the first call with that device current.  Every call on a
 * GPU shares that GPU's array: calls that overlap on one GPU (other streams,
 * other contexts, other host threads) race and give wrong results.  Other
 * errors as for rwttt_read. */
rwttt_status rwttt_read_noalloc(rwttt_ctx* ctx, const rwttt_group* group, const uint32_t* owner_map,
                                const uint64_t* expected, uint32_t layer, const void* x, void* y,
                                void* stream);

/* Tail buffers (TailBufferState, Section 4.1; TailBufferUpdate, Section 4.2
 * primitives table and "READ"): request-local update evidence, the inputs x
 * of the steps since the owner's last update boundary, kept for the next
 * WRITE.  `tail` is a host array of n_owners * n_layers device pointers
 * (index owner * n_layers + layer), each to `rows` x d_ff elements of the io
 * dtype, row-major, 16-byte aligned, owned by the caller and disjoint from
 * every other buffer.  Attaching (again) sets every tail length to 0.
 * Errors: RWTTT_E_INVALID for null or misaligned pointers or rows == 0. */
rwttt_status rwttt_attach_tail(rwttt_ctx* ctx, void* const* tail, uint32_t rows);

/* Rows currently held in the tail of (owner, layer). */
rwttt_status rwttt_tail_len(const rwttt_ctx* ctx, uint32_t owner, uint32_t layer, uint32_t* len);

/* READ with TailBufferUpdate fused (Section 4.2 primitives table, phase R):
 * rwttt_read, and in the same kernel the owner's x row is appended to the tail
 * of (owner, layer) at row tail_len, which then grows by one.  No version
 * changes (the tail is metadata, not a published state).  Errors, checked for
 * every owner before anything is launched: RWTTT_E_INVALID if no tail is
 * attached; RWTTT_E_CAPACITY if a tail is full; `expected` as for rwttt_read. */
rwttt_status rwttt_read_append(rwttt_ctx* ctx, const rwttt_group* group, const uint32_t* owner_map,
                               const uint64_t* expected, uint32_t layer, const void* x, void* y,
                               void* stream);

/* WRITE / BoundaryUpdate (Section 3, Write; Section 4.2 "WRITE"): for each
 * slot b, owner r = owner_map[first+b]:
 *     shadow_{r,layer} = live_{r,layer} + eta * Z_b^T G_b
 * with Z_b = z[b] ([chunk, d_ff]) and G_b = g[b] ([chunk, d_model]); the
 * product accumulates in fp32 and the result is rounded once to the state
 * dtype.  The adapter backend applies the same evidence to its factors, both
 * from the live (A, B):
 *     A' = A + eta * Z^T (G B^T),   B' = B + eta * (Z A)^T G
 * (the step that moves A B along Z^T G to first order), with
 * chunk <= RWTTT_ADAPTER_MAX_CHUNK.  `z` and `g` are host arrays of group.count device pointers.  The
 * group must have effect RWTTT_WRITE.
 *
 * A WRITE transition also returns the step's output (Section 3: Write_theta
 * maps (r, x_r, u_r, s_r^v) to (y_r, s_r^{v+1})): with x and y non-null
 * (owner-indexed as in rwttt_read) it also computes
 *     y[r, :] = x[r, :] W0_layer + x[r, :] live_{r,layer}
 * at version v, the candidate being invisible until commit.  For bf16
 * evidence and chunk <= 64 the token is fused into the update kernel, which
 * reads the live state once for both; otherwise the library runs a READ of
 * the group first.  Pass x = y = NULL for a WRITE without a token (prefill).
 *
 * With z == NULL the evidence rows come from the tail: the chunk is the
 * owner's tail_len rows followed by this step's own input x (the WRITE step
 * is the chunk's last token), so chunk must equal tail_len + 1 for every
 * owner and x, y must be given.  The step's x is appended to the tail first.
 *
 * Marks each owner dirty (its write view is open until commit or rollback,
 * Section 4.1).  Errors: RWTTT_E_INVALID if only one of x, y is given;
 * RWTTT_E_STALE_VERSION if `expected` (as for rwttt_read) names a version
 * other than V(r) for a member; RWTTT_E_DIRTY if this layer of an owner was
 * already written in the open transition.  If the launch fails (RWTTT_E_HIP)
 * or a failure was injected (RWTTT_E_WRITE_FAILED), the owners stay dirty and
 * are marked failed: they can only roll back. */
rwttt_status rwttt_write(rwttt_ctx* ctx, const rwttt_group* group, const uint32_t* owner_map,
                         const uint64_t* expected, uint32_t layer, uint32_t chunk,
                         const void* const* z, const void* const* g, float eta, const void* x,
                         void* y, void* stream);

/* Commit (Section 4.2 CONTROL; Algorithm 1, CommitVersions): for each owner,
 * flip the live slot of every layer written in its open transition and set
 * V(r) = V(r) + 1.  Host-only, O(owners), copies nothing.  All owners are
 * validated first: RWTTT_E_NOT_DIRTY (no candidate), RWTTT_E_WRITE_FAILED
 * (its WRITE failed), RWTTT_E_OWNER_ALIAS (listed twice).  Later launches see
 * the new live slot; they must be ordered after the WRITE on the device (same
 * stream, or an event wait).  The update boundary is closed: the owner's
 * tails become empty. */
rwttt_status rwttt_commit(rwttt_ctx* ctx, const uint32_t* owners, uint32_t n);

/* Rollback (Section 4.2 CONTROL; the failure branch of Algorithm 1): forget
 * each owner's candidate.  The live slots and V(r) are untouched, so version
 * v is restored exactly.  The chunk's evidence is dropped with it: the
 * owner's tails become empty.  Errors as for commit, except that failed
 * owners are accepted. */
rwttt_status rwttt_rollback(rwttt_ctx* ctx, const uint32_t* owners, uint32_t n);

/* View (Algorithm 1): committed version, and whether a candidate is open.
 * Either output pointer may be NULL.  Which slot is live is kept per (owner,
 * layer), since a commit flips only the layers its transition wrote, so it
 * is not an owner-wide value: rwttt_slot returns the live or shadow slot of
 * one (owner, layer). */
rwttt_status rwttt_version(const rwttt_ctx* ctx, uint32_t owner, uint64_t* version, int32_t* dirty);

/* Device address of the live (which = 0) or shadow (which = 1) slot of
 * (owner, layer) as the table stands now. */
rwttt_status rwttt_slot(const rwttt_ctx* ctx, uint32_t owner, uint32_t layer, int32_t which,
                        void** ptr);

/* Fork (Section 4.2 CONTROL: fork creates a separate owner/version lineage):
 * owner dst becomes a copy of owner src's committed state.  Every layer's
 * live slot of src (version V(src)) is copied into dst's live slot, dst's
 * tails receive src's tail rows and lengths, and V(dst) = V(src); from then
 * on the two lineages advance independently.  src may hold an open
 * candidate (it is not copied).  One kernel launch on `stream` copies all
 * layers; it reads the slots that are live at enqueue time.  Errors:
 * RWTTT_E_OWNER_ALIAS if src == dst; RWTTT_E_DIRTY if dst holds a candidate;
 * RWTTT_E_INVALID if an owner id is out of range or there is no workspace
 * (a host-only context). */
rwttt_status rwttt_fork(rwttt_ctx* ctx, uint32_t src, uint32_t dst, void* stream);

/* Checkpoint (Section 4.1 snapshot; Section 4.2 CONTROL): copy the owner's
 * committed state, the live slot of every layer (rwttt_slot_bytes bytes
 * each, in the slot layout), into dst[layer] and return its version.  dst is a
 * host array of n_layers caller-owned buffers, each pinned host memory (from
 * hipHostMalloc) or device memory; the copies are asynchronous on `stream`
 * (hipMemcpyAsync), so the caller synchronises before reading them.  An open
 * candidate is allowed and not copied.  Errors: RWTTT_E_INVALID for a bad
 * owner or a null buffer. */
rwttt_status rwttt_checkpoint(rwttt_ctx* ctx, uint32_t owner, void* const* dst,
                              uint64_t* version, void* stream);

/* Resume from a checkpoint: copy src[layer] (as written by rwttt_checkpoint)
 * into the owner's live slots, set V(owner) = version and empty its tails.
 * Asynchronous on `stream`; later launches on the same stream see the
 * restored state.  Errors: RWTTT_E_DIRTY if the owner holds a candidate;
 * RWTTT_E_INVALID for a bad owner or a null buffer. */
rwttt_status rwttt_resume(rwttt_ctx* ctx, uint32_t owner, const void* const* src,
                          uint64_t version, void* stream);

/* Failure injection for state-contract tests (Section 5.5): the next `count`
 * rwttt_write calls validate, mark their owners dirty and failed, launch
 * nothing and return RWTTT_E_WRITE_FAILED. */
rwttt_status rwttt_inject_write_failures(rwttt_ctx* ctx, uint32_t count);

/* hipError_t of the last RWTTT_E_HIP returned by this context (0 if none). */
int32_t rwttt_last_hip_error(const rwttt_ctx* ctx);

/* Static description of a status code. */
const char* rwttt_strerror(rwttt_status status);

#ifdef __cplusplus
}
#endif

#endif /* RWTTT_H */
