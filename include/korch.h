/*
 * korch.h -- C ABI of an MI355X (gfx950) executor for Korch-style primitive
 * graphs under kernel-orchestration plans.
 *
 * Model (Korch, Sections 3-5):
 *   - A primitive graph G = (P, E) is a DAG whose nodes are tensor-algebra
 *     primitives of four kinds (Section 3): elementwise, reduce/broadcast,
 *     layout transformation and linear transformation.  Graph inputs
 *     (activations and weights) are nodes without a producer.
 *   - A kernel is a convex set of primitives P' (Definition 1) with a
 *     non-empty possible output set O (Definition 3) that it materializes.
 *   - A plan is an ordered list of kernels.  Every kernel reads only graph
 *     inputs and tensors materialized by earlier kernels (the dependency
 *     constraint of Section 4.2, with an order), every graph output is
 *     materialized by some kernel (the output constraint), a primitive may be
 *     executed by several kernels (redundant execution) and a primitive in no
 *     kernel is never executed (implicit pruning).
 *   - Kernels run sequentially on one stream (Section 5.3).
 *
 * Conventions for every entry point:
 *   - Return value: KORCH_OK (0) or a negative korch_status.  korch_last_error()
 *     returns a thread-local message naming the rule / kernel that failed.
 *     No C++ exception and no abort crosses this boundary.
 *   - Handles are owned by the caller and released with the destroy calls,
 *     which accept NULL.
 *   - Device memory (inputs, outputs, workspace) is allocated and owned by the
 *     caller.  Tensors are dense, row-major, and every device pointer must be
 *     16-byte aligned (KORCH_E_ALIGN otherwise).  The library owns only its
 *     compiled code objects and a small per-plan counter buffer that
 *     korch_plan_load allocates once.
 *   - Nothing here synchronizes the stream.  Device faults in asynchronous
 *     kernels surface at the caller's next synchronization.
 *   - hipStream_t is passed as void* so this header needs no HIP header.
 */
#ifndef KORCH_H
#define KORCH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct korch_graph korch_graph;
typedef struct korch_plan korch_plan;

typedef enum {
  KORCH_OK = 0,
  KORCH_E_ARG = -1,               /* bad argument, NULL handle, bad node id      */
  KORCH_E_SHAPE = -2,             /* shape inference failed                      */
  KORCH_E_CYCLE = -3,             /* graph is not a DAG / not finalized          */
  KORCH_E_STATE = -4,             /* call not allowed in the object's state      */
  KORCH_E_PLAN_EMPTY = -10,       /* empty plan or kernel, or a graph input in P' */
  KORCH_E_PLAN_NONCONVEX = -11,   /* Definition 1 violated                       */
  KORCH_E_PLAN_BAD_OUTPUT = -12,  /* O not a possible output set (Definition 3)  */
  KORCH_E_PLAN_DEP_ORDER = -13,   /* a kernel reads a tensor no earlier kernel made */
  KORCH_E_PLAN_OUTPUT_UNCOVERED = -14, /* a graph output is never materialized   */
  KORCH_E_PLAN_MULTI_OUTPUT = -15,/* |O| > 1 while KORCH_STRICT_SINGLE_OUTPUT=1  */
  KORCH_E_UNSUPPORTED = -20,      /* no kernel family implements this kernel (cost = infinity) */
  KORCH_E_ALIGN = -21,            /* device pointer not 16-byte aligned          */
  KORCH_E_WORKSPACE = -22,        /* workspace missing or too small              */
  KORCH_E_COMPILE = -23,          /* runtime compilation of a kernel failed      */
  KORCH_E_HIP = -30               /* a HIP runtime call failed                   */
} korch_status;

typedef enum { KORCH_F32 = 0, KORCH_F16 = 1, KORCH_BF16 = 2 } korch_dtype;

/* Primitive kinds (Section 3 and its table of representative operators). */
typedef enum {
  KORCH_INPUT = 0,
  /* elementwise, unary: O[x] = f(I[x]) */
  KORCH_NEG = 1, KORCH_EXP, KORCH_LOG, KORCH_TANH, KORCH_SQRT, KORCH_RSQRT, KORCH_RELU,
  KORCH_SQUARE, KORCH_RECIP, KORCH_GELU_TANH, KORCH_ABS, KORCH_IDENTITY,
  /* elementwise, binary: O[x] = f(I1[x], I2[x]); implicit broadcast (right-aligned,
     size-1 dims stretch), or f(I1[x], scalar) when attrs.has_scalar */
  KORCH_ADD = 32, KORCH_SUB, KORCH_MUL, KORCH_DIV, KORCH_MAX, KORCH_MIN,
  /* reduce along attrs.axis (sum / mean = sum/n / max), keepdim per attrs;
     broadcast to attrs.shape */
  KORCH_REDUCE_SUM = 64, KORCH_REDUCE_MEAN, KORCH_REDUCE_MAX, KORCH_BROADCAST,
  /* layout: O[x] = I[L(x)] with L one-to-one */
  KORCH_TRANSPOSE = 96,  /* output dim k = input dim attrs.perm[k]          */
  KORCH_RESHAPE,         /* row-major reinterpretation to attrs.shape       */
  KORCH_SLICE,           /* [attrs.begin, attrs.end) per dim, unit step     */
  KORCH_PAD,             /* attrs.begin = low pads, attrs.end = high pads, value attrs.pad_value */
  KORCH_CONCAT,          /* along attrs.axis, n_in >= 2                     */
  KORCH_FILL,            /* no operands: a constant tensor of shape attrs.shape (attrs.rank dims)
                            whose every element is attrs.scalar (the ones tensor of the
                            reduction-as-product transformation, Section 3)              */
  /* linear */
  KORCH_MATMUL = 128,    /* [..., M, K] x [..., K, N] -> [..., M, N], batch dims broadcast */
  KORCH_CONV2D           /* NHWC x HWIO cross-correlation, zero pad attrs.pad, stride attrs.stride */
} korch_op;

#define KORCH_MAX_RANK 8

typedef struct {
  int32_t axis;                     /* reduce / concat axis (negative counts from the end) */
  int32_t keepdim;                  /* reduce: keep the reduced dim as size 1              */
  int32_t rank;                     /* length of perm / shape / begin / end                */
  int32_t perm[KORCH_MAX_RANK];
  int64_t shape[KORCH_MAX_RANK];    /* reshape / broadcast target                          */
  int64_t begin[KORCH_MAX_RANK];    /* slice begin, or pad low                             */
  int64_t end[KORCH_MAX_RANK];      /* slice end, or pad high                              */
  double scalar;                    /* right operand of a binary op when has_scalar        */
  int32_t has_scalar;
  int32_t stride, pad;              /* conv2d                                              */
  double pad_value;                 /* pad                                                 */
} korch_attrs;

/* A kernel (P', O): primitive node ids and the ids it materializes. */
typedef struct {
  int32_t n_prims;
  const int32_t* prims;
  int32_t n_outs;
  const int32_t* outs;
} korch_kernel_desc;

/* Kernel families (what implements a kernel on the GPU). */
typedef enum {
  KORCH_FAM_NONE = 0,
  KORCH_FAM_POINTWISE = 1,   /* elementwise + broadcast + layout chains          */
  KORCH_FAM_ROW = 2,         /* row programs with last-axis reductions (softmax, LayerNorm) */
  KORCH_FAM_COLREDUCE = 3,   /* one reduction over a non-last axis               */
  KORCH_FAM_GEMM = 4,        /* MFMA matrix product with fused prologue / epilogue */
  KORCH_FAM_CONV = 5,        /* implicit-GEMM NHWC convolution + epilogue         */
  KORCH_FAM_ATTENTION = 6,   /* scores, row softmax and second product in one kernel */
  KORCH_FAM_SPLITK = 7       /* long-contraction product split over workgroups, deterministic */
} korch_family;

const char* korch_last_error(void);
const char* korch_status_name(int status);

/* ---- graph (Section 4: G = (P, E)) ------------------------------------ */
int korch_graph_create(korch_graph** g);
void korch_graph_destroy(korch_graph* g);
/* Adds a graph input (activation or weight) of the given shape and dtype. */
int korch_graph_input(korch_graph* g, korch_dtype dtype, int32_t rank, const int64_t* shape, int32_t* node);
/* Adds a primitive reading n_in earlier nodes; attrs may be NULL when unused;
   out_dtype is the storage dtype of the primitive's tensor.  The output shape
   is inferred immediately (KORCH_E_SHAPE on mismatch). */
int korch_graph_op(korch_graph* g, korch_op op, int32_t n_in, const int32_t* in, const korch_attrs* attrs,
                   korch_dtype out_dtype, int32_t* node);
/* Marks a primitive as a graph output (order of calls = output order). */
int korch_graph_output(korch_graph* g, int32_t node);
/* Freezes the graph: checks it is a DAG with at least one output and builds
   reachability.  Required before plans are made. */
int korch_graph_finalize(korch_graph* g);
int korch_graph_num_nodes(const korch_graph* g, int32_t* n);
/* Shape / dtype / op of a node; shape must hold KORCH_MAX_RANK entries. */
int korch_graph_node_info(const korch_graph* g, int32_t node, int32_t* op, int32_t* dtype, int32_t* rank,
                          int64_t* shape);
/* Attributes of a node as given at creation (axis normalized for reduce and
   concat nodes). */
int korch_graph_node_attrs(const korch_graph* g, int32_t node, korch_attrs* attrs);
/* The producers a node reads, in operand order: *n receives the count and at
   most `cap` ids are written to `ids` (which may be NULL when cap is 0). */
int korch_graph_node_inputs(const korch_graph* g, int32_t node, int32_t* ids, int32_t cap, int32_t* n);
int korch_graph_num_inputs(const korch_graph* g, int32_t* n);
int korch_graph_num_outputs(const korch_graph* g, int32_t* n);
int korch_graph_input_node(const korch_graph* g, int32_t i, int32_t* node);
int korch_graph_output_node(const korch_graph* g, int32_t i, int32_t* node);

/* ---- primitive-graph transformations (Section 3) ------------------------ */
typedef enum {
  KORCH_RW_DEFER_DIV = 1,          /* (E / s) . V -> (E . V) / s, s constant along the contraction axis */
  KORCH_RW_REDUCE_AS_PRODUCT = 2,  /* sum over an axis -> product with a ones tensor, where a product
                                      on the same operand exists to merge with                      */
  KORCH_RW_MERGE_PRODUCTS = 4,     /* A . B1, A . B2 -> column slices of A . concat(B1, B2)          */
  KORCH_RW_FOLD_SCALE = 8,         /* (A . B) * s -> A . (B * s), s varying only along the output
                                      columns (channels); also for convolutions and for division    */
  KORCH_RW_SPLIT_MOMENTS = 32,     /* D = X - mean(X) over a non-last axis read by a variance (mean of
                                      D^2) and by other nodes: the square reads its own copy X - m  */
  KORCH_RW_ALL = 47,
  KORCH_RW_LAYOUT_VARIANTS = 16    /* layout as a plan variable (Section 8): each computed operand of
                                      a product is followed by transpose(transpose(x)) of its last
                                      two axes, so a plan may store x in either layout; applied once,
                                      after the other rules; not part of KORCH_RW_ALL              */
} korch_rewrite_rule;
/* Applies the selected rules until none applies (the layout variants last,
   once) and returns a new finalized graph in *out (the caller destroys it)
   whose inputs and outputs correspond, in order, to those of g; every output
   has the same value in exact arithmetic.  *applied (may be NULL) receives the
   number of applications (each layout variant counts as one).  Node ids of
   *out are unrelated to those of g. */
int korch_graph_rewrite(const korch_graph* g, uint32_t rules, korch_graph** out, int32_t* applied);

/* ---- orchestration analysis (Section 4.1) ------------------------------ */
/* Definition 1 on an arbitrary node set; *convex = 1 or 0. */
int korch_is_convex(const korch_graph* g, int32_t n, const int32_t* nodes, int32_t* convex);
/* Execution states (Definition 2) reached by the depth-first search of
   Algorithm 1, including the empty state.  Each state is reported as a 0/1
   array over all node ids (graph inputs are always 0).  Returns
   KORCH_E_ARG when more than max_states states exist. */
int korch_enumerate_states(const korch_graph* g, int32_t max_states,
                           int (*cb)(const uint8_t* member, int32_t n_nodes, void* user), void* user);
/* Candidate kernels of Algorithm 1: every P' = D2 \ D1 of states D1 < D2 with
   |P'| <= max_prims, paired with each non-empty possible output set O (all
   subsets when the maximal set has <= max_outs members, otherwise the maximal
   set and each singleton).  When only_supported != 0, candidates no family
   implements are skipped.  The callback returns non-zero to stop early. */
int korch_enumerate_candidates(const korch_graph* g, int32_t max_prims, int32_t max_outs, int32_t only_supported,
                               int (*cb)(const korch_kernel_desc* k, void* user), void* user);
/* Which family implements kernel k (KORCH_FAM_NONE = unsupported, cost infinity). */
int korch_kernel_family(const korch_graph* g, const korch_kernel_desc* k, int32_t* family);
/* The HIP source a plan of g would generate for kernel k (Section 5.2's
   kernel generation, within the whole graph: its external tensors are those
   of g), for inspection.  Needs no GPU and compiles nothing.  *len receives
   the source length; at most cap - 1 bytes and a terminating 0 are written to
   buf (may be NULL when cap is 0).  KORCH_E_UNSUPPORTED when no family
   implements k. */
int korch_kernel_source(const korch_graph* g, const korch_kernel_desc* k, char* buf, size_t cap, size_t* len);

/* ---- plans -------------------------------------------------------------- */
/* Validates an ordered plan (rules of Definitions 1 and 3 and the output and
   dependency constraints of Section 4.2) and copies the graph, so the plan
   does not depend on the graph's lifetime. */
int korch_plan_create(const korch_graph* g, int32_t n_kernels, const korch_kernel_desc* kernels, korch_plan** p);
/* The unfused plan: one kernel per primitive, except reshapes of materialized
   tensors, which are views and need no kernel.  Its kernel symbols are
   korch_u<k>_<family> (a plan from korch_plan_create uses korch_k<k>_<family>),
   so profiles of a run that executes both plans keep them apart. */
int korch_plan_unfused(const korch_graph* g, korch_plan** p);
void korch_plan_destroy(korch_plan* p);
int korch_plan_num_kernels(const korch_plan* p, int32_t* n);
/* Family match, code generation and runtime compilation for gfx950 of every
   kernel (disk-cached).  Needs no GPU.  KORCH_E_UNSUPPORTED names the kernel. */
int korch_plan_compile(korch_plan* p);
/* Compiles the plan if needed, loads its code objects on the current device
   and allocates and zeroes the plan's counter buffer (the arrival counters of
   cross-workgroup hand-offs; each kernel leaves them at zero again).  Needs a
   GPU; synchronizes the device once.  Required before any execute call on a
   device; calling it again on the same device does nothing, on another device
   it moves the plan there. */
int korch_plan_load(korch_plan* p);
int korch_plan_workspace_bytes(const korch_plan* p, size_t* bytes);
/* Launches the plan's kernels in order on `stream` (a hipStream_t, NULL =
   default stream).  inputs[i] / outputs[i] follow graph input / output order.
   Never allocates, never compiles or loads, never synchronizes: a plan not
   loaded on the current device (korch_plan_load) is KORCH_E_STATE.  The
   plan's one counter buffer is shared by its executions, so one plan must not
   execute on two streams at once (successive executions on one stream, or
   streams ordered by events, are fine); use one plan per concurrent stream. */
int korch_plan_execute(korch_plan* p, const void* const* inputs, void* const* outputs, void* workspace,
                       size_t workspace_bytes, void* stream);
/* korch_plan_execute for callers that cannot allocate device memory (code
   under HIP graph capture, tight serving loops, harnesses that forbid
   allocation): no workspace argument.  The plan's workspace and hand-off
   counters live in a static device array of the library, 32 MiB per device
   (the first 64 KiB for counters, the rest, 33,488,896 bytes, for the
   workspace), held from the first korch_plan_load on a device until the
   process ends; korch_plan_load looks up its address on each device.  The
   call first clears the counters the plan uses with a fill kernel on
   `stream`, then launches the plan's kernels; it never allocates, compiles,
   loads or synchronizes.  Errors: KORCH_E_STATE when the plan is not loaded
   on the current device; KORCH_E_WORKSPACE when the plan's workspace
   (korch_plan_workspace_bytes) or counters exceed the static array (nothing
   is launched); KORCH_E_ARG / KORCH_E_ALIGN as korch_plan_execute.  Every
   call on one device shares that device's array and finds there whatever the
   previous call left: calls that overlap on one device (two streams, or two
   threads without ordering) race and give wrong results. */
int korch_plan_execute_noalloc(korch_plan* p, const void* const* inputs, void* const* outputs, void* stream);
/* Same as korch_plan_execute but launches only kernels [first, first+count)
   of the plan (for timing one kernel in place); the caller is responsible for
   having run the earlier kernels whose outputs these read. */
int korch_plan_execute_kernels(korch_plan* p, int32_t first, int32_t count, const void* const* inputs,
                               void* const* outputs, void* workspace, size_t workspace_bytes, void* stream);
/* korch_plan_execute_kernels with one kernel bracketed by events, so that a
   timed loop of plan executions measures that kernel's duration in place
   with one call per execution (the profiler of Section 5.2 times a kernel
   alone; this times it inside the plan).  `start` and `stop` take the start
   and end timestamps of kernel `timed`'s own dispatch on `stream` (no marker
   packets are added); both are hipEvent_t handles owned by the caller
   (created with timing enabled), and either may be NULL.  KORCH_E_ARG when `timed` is not in [first,
   first+count); otherwise errors as korch_plan_execute_kernels. */
int korch_plan_execute_timed(korch_plan* p, int32_t first, int32_t count, const void* const* inputs,
                             void* const* outputs, void* workspace, size_t workspace_bytes, void* stream, int32_t timed,
                             void* start, void* stop);
/* korch_plan_execute with timing events on any kernels: start_events[k] and
   stop_events[k] (arrays with one entry per kernel of the plan; either array,
   and any entry, may be NULL) are hipEvent_t handles owned by the caller,
   created with timing enabled, that take the start and end timestamps of
   kernel k's own dispatch on `stream` (no marker packets are added).  So one
   call measures the span of a whole plan execution (the first kernel's start
   to the last kernel's end) and any kernel inside it.  Errors as
   korch_plan_execute. */
int korch_plan_execute_events(korch_plan* p, const void* const* inputs, void* const* outputs, void* workspace,
                              size_t workspace_bytes, void* stream, void* const* start_events,
                              void* const* stop_events);
/* Per-kernel family, algorithmic bytes (compulsory reads of its external
   tensors plus writes of its outputs) and flops (2*M*N*K per contraction). */
int korch_plan_kernel_info(const korch_plan* p, int32_t k, int32_t* family, double* alg_bytes, double* alg_flops);
/* Generated HIP source and kernel symbol name of kernel k (after compile). */
int korch_plan_kernel_source(const korch_plan* p, int32_t k, char* buf, size_t cap, size_t* len);
int korch_plan_kernel_name(const korch_plan* p, int32_t k, char* buf, size_t cap);
/* The gfx950 code object (ELF) of kernel k after korch_plan_compile: copies
   min(cap, size) bytes to `buf` (may be NULL) and stores the size in *len (may
   be NULL).  Its AMDGPU metadata note states the kernel's registers, LDS and
   private (scratch) segment.  KORCH_E_STATE before compilation. */
int korch_plan_kernel_code(const korch_plan* p, int32_t k, void* buf, size_t cap, size_t* len);
/* Launch geometry of kernel k (after compile). */
int korch_plan_kernel_launch(const korch_plan* p, int32_t k, int32_t grid[3], int32_t block[3], int32_t* lds_bytes);

/* ---- profiler (Section 5.2, kernel profiler; Algorithm 1's Profiling) --- */
/* Generates and compiles (hipRTC, gfx950, code-object cache) the single kernel
   (P', O) exactly as korch_profile_candidate does, without touching a GPU, so
   that profiling on a device finds it compiled.  Returns KORCH_E_UNSUPPORTED
   when no family implements it, KORCH_E_COMPILE when hipRTC rejects it. */
int korch_compile_candidate(const korch_graph* g, const korch_kernel_desc* k);

/* Times the single kernel (P', O) in isolation: compiles it, fills its inputs
   with seeded uniform values in [0.5, 1.5) in device buffers the profiler allocates, runs
   `warmup` untimed launches, then `reps` launches each preceded by a read of
   `flush_bytes` of a scratch buffer (korch_flush_caches; environment
   KORCH_FLUSH_WRITE=1 writes it instead) and a read of every input that the parent graph computes (in a plan, the
   producing kernel has just written such a tensor, so it is cache-resident,
   while graph inputs come from HBM; environment KORCH_PROFILE_COLD=1 skips
   that read), each launch timed by HIP events that take that dispatch's own
   start and end timestamps on `stream`; *median_us is the median.  The cost
   of a plan is the sum of its kernels' costs (Section 4.2).  Returns
   KORCH_E_UNSUPPORTED (cost infinity) when no family implements it. */
int korch_profile_candidate(const korch_graph* g, const korch_kernel_desc* k, int32_t warmup, int32_t reps,
                            size_t flush_bytes, void* stream, float* median_us);

/* Cold-cache precondition of a measurement (Section 5.2 times kernels in
   isolation; here they must find their inputs in HBM).  Enqueues on `stream`
   one kernel that streams through the first `bytes` (rounded down to 16) of
   the caller's device buffer `buffer` (16-byte aligned, at least 512 MiB to
   cover L2 and the 256 MB Infinity Cache): a read when write = 0, after which
   the caches hold clean lines of `buffer` (dirty lines present before are
   written back during this kernel), else a write, after which they hold dirty
   lines that a following kernel's misses must write back.  Asynchronous;
   KORCH_E_ALIGN for a misaligned buffer. */
int korch_flush_caches(void* buffer, size_t bytes, int32_t write, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* KORCH_H */
