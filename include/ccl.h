/*
 * ccl.h - GEMM on operands stored in Chiplet-Contiguous Layout (CCL),
 *         for AMD Instinct MI355X (gfx950).
 *
 * Method: "Making Locality-aware GEMM Compatible with Page-Granularity
 * Placement on Chiplet GPUs" (Chung, Ju, Kim).
 *   - C = A B with A (M x K), B (K x N), C (M x N), Sec. II-B.
 *   - Each chiplet's operand share is one contiguous, page-aligned strip:
 *     Sec. III-B, Eq. 1-3 (CCL index g*K*w + k*w + n'), Sec. III-C.
 *   - Output tiles run on the chiplet that owns them (Sec. III-A) and the
 *     GEMM arithmetic itself is unchanged (Sec. III-C).
 *   - Remote-HBM traffic under 4 KB round-robin interleave, coarse
 *     locality-aware placement and CCL, Sec. IV-A.
 *
 * Conventions for every call:
 *   - Element types are the plan's: bfloat16 (2 bytes) for A, B and C with
 *     ccl_plan (Sec. IV-A: BF16 GEMMs); ccl_plan_typed also takes fp8 E4M3
 *     A and B and an fp32 C (Fig. 7 data types). e below is the element
 *     size in bytes. Device buffers are passed as plain device pointers.
 *   - Logical operands are row-major: A is M x K, B is K x N, C is M x N.
 *   - The caller owns every buffer and the stream. The library allocates no
 *     device memory. A plan is owned by the caller from ccl_plan() until
 *     ccl_plan_destroy(); it is immutable, so calls on one plan may run from
 *     several host threads.
 *   - Device calls (ccl_pack, ccl_unpack, ccl_gemm, ccl_debug_dispatch) are
 *     asynchronous on `stream` (a hipStream_t passed as void*; NULL is the
 *     null stream). ccl_plan*, ccl_remote_bytes and ccl_debug_tile_of_wg are
 *     host-only and need no GPU.
 *   - Every call returns a ccl_status. On any error nothing is written and
 *     nothing is launched; ccl_last_error() gives a per-thread message.
 *   - Tuning overrides, read when a plan is made: CCL_GEMM_TILE=RxC (kernel
 *     tile 256x256, 256x128, 128x256 or 128x128), CCL_GEMM_WAVES=4|8 (waves
 *     per workgroup; 8, the default, exists for every bf16 tile and for fp8
 *     256x256 tiles) and CCL_GEMM_GROUP_M=n (rows of the tile raster group).
 *     Unset, the plan chooses.
 *
 * CCL layout of an operand X (R x Cc) under a Gr x Gc grid (the same grid
 * is laid over each operand's own rows and columns: A is split along K by
 * Gc, B along K by Gr):
 *   hr = R / Gr, wc = Cc / Gc, block b(r, c) = (r / hr) * Gc + c / wc,
 *   strip bytes S = ceil(hr * wc * e / page) * page,
 *   byte offset(r, c) = b * S + ((r % hr) * wc + c % wc) * e.
 * Block b lives on chiplet b. With Gr = 1 and no padding this is Eq. 3.
 * Padding bytes at the end of each strip are never read or written.
 */
#ifndef CCL_H_
#define CCL_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ccl_plan_s* ccl_plan_t;

typedef enum {
  CCL_OK = 0,
  CCL_ERR_INVALID_ARG = 1,          /* bad size, grid, page, operand, null pointer */
  CCL_ERR_UNALIGNED_PARTITION = 2,  /* partitions not multiples of the 128x128 tile */
  CCL_ERR_UNSUPPORTED = 3,          /* valid plan the GPU path does not run */
  CCL_ERR_MISALIGNED_POINTER = 4,   /* device pointer / leading dimension alignment */
  CCL_ERR_HIP = 5                   /* HIP runtime error (launch, device query) */
} ccl_status;

typedef enum { CCL_A = 0, CCL_B = 1, CCL_C = 2 } ccl_operand;

/* Element types (Fig. 7 sweeps the data type). A and B share one type. */
typedef enum {
  CCL_DT_BF16 = 0,       /* 2 bytes */
  CCL_DT_FP8_E4M3 = 1,   /* 1 byte: OCP 8-bit float, 4 exponent bits (bias 7), 3 mantissa bits */
  CCL_DT_FP32 = 2        /* 4 bytes (C; A and B for layouts and traffic models) */
} ccl_dtype;

typedef enum {
  CCL_PLACE_RR = 0,      /* fixed-size pages to chiplets round-robin (Sec. IV-A) */
  CCL_PLACE_COARSE = 1,  /* G contiguous page-granular chunks (Sec. IV-A, Coarse LA) */
  CCL_PLACE_CCL = 2      /* CCL strips, each strip's pages on its chiplet */
} ccl_placement;

/* Layout of one operand in CCL. All sizes in elements unless named _bytes. */
typedef struct {
  int64_t rows, cols;            /* logical operand shape */
  int64_t grid_r, grid_c;        /* block grid over (rows, cols) */
  int64_t block_rows, block_cols;
  int64_t strip_bytes;           /* block_rows * block_cols * 2 */
  int64_t strip_stride_bytes;    /* strip_bytes rounded up to the page */
  int64_t total_bytes;           /* grid_r * grid_c * strip_stride_bytes: buffer size */
  int64_t elem_bytes;            /* bytes per element: 1 (fp8), 2 (bf16) or 4 (fp32) */
} ccl_layout;

#define CCL_MAX_CHIPLETS 64

/* Remote-byte record (Sec. IV-A metric, no cache): every 128x128 output
 * tile runs on its owner chiplet, reads its full A row panel and B column
 * panel and writes its C tile; an access is remote iff its page is on
 * another chiplet. Index [0]=A, [1]=B, [2]=C. */
typedef struct {
  uint64_t accessed[3];          /* bytes read (A, B) or written (C) */
  uint64_t remote[3];            /* of which remote */
  uint64_t floor_bytes;          /* lower bound of remote bytes for any layout */
  uint64_t footprint[3];         /* stored bytes of each operand, padding included */
  uint64_t remote_per_chiplet[CCL_MAX_CHIPLETS];  /* charged to the requesting owner */
  int32_t chiplets;
} ccl_traffic;

/*
 * Create a plan for C = A B over `chiplets` chiplets (1..64) on a
 * grid_rows x (chiplets / grid_rows) output-partition grid, with strips
 * padded to `page_bytes` (power of two, >= 128). grid_rows = 0 chooses the
 * grid per GEMM (Sec. IV-A "Baselines": CCL picks coarse or fine
 * partitioning per GEMM): the tile-aligned grid with the fewest CCL remote
 * bytes, then the one whose shared operands replicate fewer bytes, then the
 * smaller grid_rows.
 * All three operands are bf16 (ccl_plan_typed with CCL_DT_BF16, CCL_DT_BF16).
 * Errors: CCL_ERR_INVALID_ARG (non-positive size, chiplets out of range,
 * grid_rows not dividing chiplets, bad page, out == NULL, size overflow);
 * CCL_ERR_UNALIGNED_PARTITION (M % (Gr*128), N % (Gc*128), K % Gr or
 * K % Gc not zero, or no aligned grid for grid_rows = 0).
 */
ccl_status ccl_plan(int64_t M, int64_t N, int64_t K, int chiplets, int grid_rows,
                    int64_t page_bytes, ccl_plan_t* out);

/*
 * ccl_plan with element types: ab_type for A and B (CCL_DT_BF16 or
 * CCL_DT_FP8_E4M3; CCL_DT_FP32 is accepted for layouts, pack/unpack and the
 * traffic models, while ccl_gemm returns CCL_ERR_UNSUPPORTED for it), c_type
 * for C (CCL_DT_BF16 or CCL_DT_FP32). The element
 * size sets the strip bytes and padding of each layout and the bytes of the
 * traffic models (Sec. II-B: the slice a chiplet needs is N/G elements, so
 * its byte size depends on the type). The automatic grid weighs A and B by
 * their element size. Errors as ccl_plan; CCL_ERR_INVALID_ARG also for
 * other type combinations.
 */
ccl_status ccl_plan_typed(int64_t M, int64_t N, int64_t K, int chiplets, int grid_rows,
                          int64_t page_bytes, ccl_dtype ab_type, ccl_dtype c_type,
                          ccl_plan_t* out);

/* Release a plan. NULL is accepted. */
ccl_status ccl_plan_destroy(ccl_plan_t plan);

/* Grid the plan uses (after automatic choice). */
ccl_status ccl_plan_grid(ccl_plan_t plan, int* grid_rows, int* grid_cols);

/* Layout of operand `op`: buffer size and strip geometry (Sec. III-B). */
ccl_status ccl_plan_layout(ccl_plan_t plan, ccl_operand op, ccl_layout* out);

/*
 * Pack a stored operand into CCL (Sec. III-C: weights packed at load time,
 * activations repacked). src_trans = 0: src is the row-major operand
 * (rows x cols, leading dimension ld >= cols elements). src_trans = 1: src
 * holds the transpose (cols x rows, ld >= rows), e.g. H for A = H^T.
 * Elements are the operand's type (bit copies, any of the three types).
 * dst_ccl has ccl_plan_layout().total_bytes bytes; padding is not written.
 * Errors: CCL_ERR_INVALID_ARG (null pointer, op not A/B/C, ld too small,
 * src_trans on C); CCL_ERR_HIP.
 */
ccl_status ccl_pack(ccl_plan_t plan, ccl_operand op, const void* src, int64_t ld,
                    int src_trans, void* dst_ccl, void* stream);

/*
 * Inverse of ccl_pack with src_trans = 0: CCL buffer -> row-major operand
 * (rows x cols, leading dimension ld >= cols). This is the inverse of the
 * Eq. 3 map (Sec. III-B: each CCL index names exactly one element of the
 * row-major matrix of Eq. 2), used where a CCL result, e.g. the output C of
 * Sec. III-C, is handed to code that expects row-major. src_ccl has
 * ccl_plan_layout().total_bytes bytes; its padding is not read. Columns
 * beyond cols in each dst row are not written. Errors as ccl_pack.
 */
ccl_status ccl_unpack(ccl_plan_t plan, ccl_operand op, const void* src_ccl, void* dst,
                      int64_t ld, void* stream);

/*
 * C_ccl = A_ccl B_ccl, all three in the plan's CCL layouts: bf16 or fp8
 * E4M3 inputs (the plan's A/B type), fp32 accumulation on the matrix cores,
 * output rounded to nearest even to bf16 or stored as fp32, per the plan's C
 * type (Sec. II-B, III-C; Fig. 7 data types). Each XCD computes exactly the output tiles of
 * the partition its chiplet owns (chiplet c <-> XCDs c*8/G .. c*8/G+8/G-1),
 * so chiplets must divide 8.
 * Errors: CCL_ERR_INVALID_ARG (null pointer); CCL_ERR_MISALIGNED_POINTER
 * (pointer not 16-byte aligned); CCL_ERR_UNSUPPORTED (chiplets not dividing
 * 8, K / Gc or K / Gr not a multiple of 32 for bf16 or of 64 for fp8,
 * device not gfx950); CCL_ERR_HIP.
 */
ccl_status ccl_gemm(ccl_plan_t plan, const void* A_ccl, const void* B_ccl, void* C_ccl,
                    void* stream);

/*
 * C_ccl = alpha * A_ccl B_ccl + beta * C_ccl, the BLAS form of the GEMM
 * (Sec. II-B): the scalars change no placement, and each output tile's owner
 * reads its C tile where it writes it. The product is accumulated in fp32,
 * then alpha * acc + beta * c is formed in fp32 and stored in C's type
 * (bf16: nearest even). beta == 0: C is not read (its old contents, NaN included, do not
 * matter), as in BLAS. ccl_gemm is alpha = 1, beta = 0.
 * Errors as ccl_gemm.
 */
ccl_status ccl_gemm_scaled(ccl_plan_t plan, float alpha, const void* A_ccl, const void* B_ccl,
                           float beta, void* C_ccl, void* stream);

/*
 * Split-K form of ccl_gemm_scaled, for GEMMs whose partitions have fewer
 * output tiles than an XCD has compute units (small M x N, long K: e.g. the
 * weight gradients of Sec. IV-A). Not a method of the paper: the ownership of
 * Sec. II-B is kept, as every K range of a tile, its fp32 partial and the
 * reduction that writes the tile all run on XCDs of the chiplet owning it.
 *
 * ccl_gemm_splitk_workspace: in: *splits = the requested number of K
 * ranges per tile (1..16), or 0 to let the library choose (enough ranges to
 * give each of an XCD's 32 compute units a workgroup, each range at least 8
 * main-loop steps). out: *splits = the number of non-empty ranges actually
 * used (the K steps, 32 bf16 or 64 fp8 elements each, are cut into ranges
 * of ceil(steps / requested)), *workspace_bytes = the device workspace that
 * ccl_gemm_splitk needs for that request: G * tiles * ranges * tile_m *
 * tile_n * 4 bytes, 0 when one range is used.
 *
 * ccl_gemm_splitk: C_ccl = alpha * A_ccl B_ccl + beta * C_ccl as
 * ccl_gemm_scaled, with `splits` as requested above. With more than one
 * range, two kernels run in order on `stream`: the K ranges write fp32
 * partial tiles to `workspace` (caller-owned device memory, 16-byte
 * aligned, at least the size reported for the same plan and splits; its
 * contents on entry do not matter and are left undefined), then each tile's
 * partials are summed in ascending range order in fp32 and alpha * sum +
 * beta * c is stored in C's type. One range: exactly ccl_gemm_scaled, and
 * the workspace is not used (may be NULL). Calls that share a workspace
 * must be ordered on one stream.
 * Errors: as ccl_gemm_scaled; CCL_ERR_INVALID_ARG also for NULL splits or
 * workspace_bytes, splits outside 0..16 (workspace query) or 1..16 (GEMM),
 * or a NULL or too small workspace when more than one range is used;
 * CCL_ERR_MISALIGNED_POINTER for a workspace not 16-byte aligned;
 * CCL_ERR_UNSUPPORTED when the split grid would exceed 2^31 workgroups.
 */
ccl_status ccl_gemm_splitk_workspace(ccl_plan_t plan, int* splits, int64_t* workspace_bytes);
ccl_status ccl_gemm_splitk(ccl_plan_t plan, float alpha, const void* A_ccl, const void* B_ccl,
                           float beta, void* C_ccl, int splits, void* workspace,
                           int64_t workspace_bytes, void* stream);

/*
 * ccl_gemm_splitk without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). The fp32 partial tiles go to a static
 * device array inside the library, CCL_SCRATCH_BYTES per GPU, reserved when
 * the library's code is loaded on that GPU and held until the process ends;
 * the call allocates nothing. Same arithmetic, kernels and results as
 * ccl_gemm_splitk with the same plan and splits. The array is shared by
 * every call on one GPU and keeps the last call's partials (nothing in it
 * has to start at zero): calls that may overlap on one GPU (different
 * streams, several host threads) race and must be ordered by the caller.
 * One range (splits such that a single K range results): exactly
 * ccl_gemm_scaled, the array is not used.
 * Errors: as ccl_gemm_splitk; CCL_ERR_INVALID_ARG also when the workspace
 * the plan and splits need (ccl_gemm_splitk_workspace) exceeds
 * CCL_SCRATCH_BYTES, checked before any device call.
 */
#define CCL_SCRATCH_BYTES (64LL << 20)
ccl_status ccl_gemm_splitk_noalloc(ccl_plan_t plan, float alpha, const void* A_ccl,
                                   const void* B_ccl, float beta, void* C_ccl, int splits,
                                   void* stream);

/*
 * Baseline for comparison with ccl_gemm (the layout the paper starts from,
 * Sec. II-B Eq. 2): the same GEMM kernel on plain row-major operands
 * A (M x K), B (K x N) and C (M x N), leading dimensions K, N and N, with
 * the plan's tile grid. remap = 1 sends every tile to an XCD of the chiplet
 * owning its partition, as ccl_gemm does; remap = 0 keeps the native
 * dispatch order (workgroup w computes the w-th tile of a grouped raster
 * over all of C and runs on XCD w mod 8, whoever owns the tile).
 * Errors as ccl_gemm; CCL_ERR_INVALID_ARG also for remap not 0 or 1.
 */
ccl_status ccl_gemm_rowmajor(ccl_plan_t plan, const void* A, const void* B, void* C, int remap,
                             void* stream);

/* Flags of ccl_remote_bytes and ccl_remote_bytes_l2. */
#define CCL_TRAFFIC_A_TRANS 1   /* A is stored transposed (e.g. H held for A = H^T) */
#define CCL_TRAFFIC_B_TRANS 2   /* B is stored transposed */
#define CCL_TRAFFIC_C_READ 4    /* C is read as well as written: alpha A B + beta C,
                                   beta != 0 (Sec. II-B: the read is partitioned
                                   like the write, so each tile's owner reads it) */

/*
 * Remote-byte record of the plan's GEMM under `placement` (Sec. IV-A).
 * flags: CCL_TRAFFIC_* bits. The stored-transpose bits affect RR and COARSE
 * only (they place pages of the stored tensor); CCL_TRAFFIC_C_READ charges
 * each C tile a read as well as the write. Host-only, synchronous.
 * Errors: CCL_ERR_INVALID_ARG (NULL argument, bad placement, flags outside 0..7).
 */
ccl_status ccl_remote_bytes(ccl_plan_t plan, ccl_placement placement, int flags,
                            ccl_traffic* out);

/* Private L2 of each chiplet for ccl_remote_bytes_l2 (Sec. IV-A: the
 * paper's configuration is 8 MB, 128-byte lines, 16-way per chiplet). */
typedef struct {
  int64_t l2_bytes;   /* capacity per chiplet; 0 = no cache. Otherwise a power-of-two
                         number of sets of ways * line_bytes, and l2_bytes / line_bytes <= 2^24 */
  int32_t ways;       /* associativity, >= 1 */
  int32_t line_bytes; /* power of two, 16 .. page_bytes */
  int32_t slots;      /* tiles a chiplet runs at once (its CTA concurrency), >= 1 */
  int32_t k_step;     /* K elements every resident tile reads per step, >= 1 */
  int32_t traversal;  /* order of a chiplet's tiles: 0 tile rows outer, 1 tile columns outer,
                         2 grouped raster (the partition's tile rows in groups of group_rows,
                         the last one possibly shorter; each group walked column by column
                         down its rows, as the GEMM kernel's workgroup map does) */
  int32_t threads;    /* host threads (capped at the core count); 0 = one per chiplet,
                         up to the core count. Each thread holds one chiplet's tags:
                         l2_bytes / line_bytes * 8 bytes of host memory. */
  int32_t group_rows; /* traversal 2: tile rows per group, >= 1; ignored otherwise */
} ccl_l2_config;

/* Result of ccl_remote_bytes_l2. Index [0]=A, [1]=B, [2]=C. */
typedef struct {
  uint64_t accesses[2];          /* L2 line accesses of A and B */
  uint64_t misses[2];            /* of which missed */
  uint64_t remote[3];            /* bytes: remote misses * line_bytes (A, B); C lines written
                                    to another chiplet * line_bytes */
  uint64_t remote_per_chiplet[CCL_MAX_CHIPLETS];  /* charged to the chiplet running the tile */
  int32_t chiplets;
} ccl_l2_traffic;

/*
 * Remote-HBM traffic of the plan's GEMM with a private set-associative LRU L2
 * per chiplet (Sec. IV-A simulation framework and metric; Fig. 7 sweeps the
 * capacity). Model:
 *   - chiplet p runs the 128x128 tiles of its partition in `traversal` order,
 *     `slots` at a time; the tiles of such a wave step through K together,
 *     k_step at a time, and at each step each tile (in wave order) reads the
 *     lines of its A slice (128 x k_step) and then of its B slice
 *     (k_step x 128), each in increasing address order of the operand as
 *     stored (row-major, stored transposed per the flags, or CCL);
 *   - A is at address 0, B at 2^40, C at 2^41; a line's set is its line
 *     number XOR-folded into log2(sets) bits; replacement is LRU;
 *   - a miss is remote when the line's home chiplet under `placement` (as in
 *     ccl_remote_bytes) is not p; after a wave, its C tiles are written
 *     (and first read, with CCL_TRAFFIC_C_READ) without allocating in L2,
 *     and every C line homed elsewhere counts each time.
 * With l2_bytes = 0 and line-aligned slices the result equals
 * ccl_remote_bytes. Host-only, synchronous; runs one host thread per chiplet.
 * Errors: CCL_ERR_INVALID_ARG (NULL argument, bad placement, flags outside
 * 0..7, invalid configuration).
 */
ccl_status ccl_remote_bytes_l2(ccl_plan_t plan, ccl_placement placement, int flags,
                               const ccl_l2_config* config, ccl_l2_traffic* out);

/* Static name of a status code. */
const char* ccl_status_string(ccl_status status);

/* Detail of the last error on the calling thread ("" if none). */
const char* ccl_last_error(void);

/*
 * Test hook: which XCD runs workgroup `wg` of ccl_gemm's launch (dispatch
 * is round-robin: wg mod 8) and which kernel output tile (tile_m, tile_n)
 * it computes, in units of the kernel tile (tile_rows x tile_cols, see
 * ccl_debug_gemm_config); -1 for both when the workgroup has no tile.
 */
ccl_status ccl_debug_tile_of_wg(ccl_plan_t plan, int64_t wg, int* xcd, int64_t* tile_m,
                                int64_t* tile_n);

/* Test hook: the GEMM kernel tile and launch size the plan uses. */
ccl_status ccl_debug_gemm_config(ccl_plan_t plan, int* tile_rows, int* tile_cols,
                                 int64_t* workgroups);

/*
 * Profiling hook: ccl_gemm (same kernel, same C) on a bf16 plan, with each
 * wave of every workgroup that has a tile recording its phase timeline.
 * `timeline` is a device buffer of at least workgroups * waves * 64 bytes
 * (ccl_debug_gemm_config gives the workgroups; waves per workgroup is 8,
 * or 4 under CCL_GEMM_WAVES=4), 16-byte aligned, owned by the caller.
 * Wave v of workgroup w writes 8 uint64 at index (w * waves + v) * 8:
 *   0-3  the 100 MHz real-time counter at its start, after the prologue
 *        (first stages in LDS), after the K loop and after its C stores
 *        were issued (they complete after the wave ends, as in ccl_gemm);
 *   4-5  the shader clock counter at its start and after the K loop;
 *   6    the XCD id it ran on; 7 the raw HW_ID register (CU, SH, SE).
 * Entries of workgroups without a tile are not written. Errors as
 * ccl_gemm; CCL_ERR_UNSUPPORTED for fp8 plans; CCL_ERR_INVALID_ARG for a
 * NULL or short timeline.
 */
ccl_status ccl_debug_gemm_timeline(ccl_plan_t plan, const void* A_ccl, const void* B_ccl,
                                   void* C_ccl, uint64_t* timeline, int64_t timeline_bytes,
                                   void* stream);

/*
 * Test hook: launch a kernel with ccl_gemm's grid in which every workgroup
 * records, at out[4*wg .. 4*wg+3], the hardware XCD id it ran on, its tile
 * (tile_m, tile_n; -1 if none) and the chiplet owning that tile. `out` is a
 * device buffer of 4 * workgroups int32. Errors as ccl_gemm.
 */
ccl_status ccl_debug_dispatch(ccl_plan_t plan, int32_t* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CCL_H_ */
