/*
 * Fused attention forward for AMD MI355X (gfx950 / CDNA4): C ABI.
 *
 * The library computes O = softmax(scale * Q K^T) V per (batch, head) as two
 * chained matrix-core products with an online softmax between them, so the
 * L x L score matrix never reaches device memory (paper: Section 6, the
 * attention equation, Algorithm 1 and Figure 2).  Tile sizes come from a
 * closed-formula derivation over a hardware descriptor (Sections 3 and 4,
 * Table 2); nothing is searched or tuned at run time.
 *
 * Conventions for every entry point:
 *  - Return value: 0 (ATTN_OK) on success, a negative attn_status_t on error.
 *    attn_strerror() names the code.  Arguments are validated before any HIP
 *    call is made, so a rejected call has no device side effect.
 *  - Tensors Q, K, V, O: device pointers to contiguous [B, H, L, d] arrays
 *    (d innermost), element type given by `dtype`; each (b, h) slice is the
 *    paper's row-major L x d matrix.  O has the same type as the inputs.
 *    Every tensor base address must be 16-byte aligned.
 *  - The caller owns every buffer it passes.  Calls are asynchronous: they
 *    enqueue work on `stream` (a hipStream_t; NULL is the null stream) and
 *    return without synchronising.  Inputs must stay valid until that work
 *    completes.
 *  - Sizes: 1 <= B, H; 1 <= L <= ATTN_MAX_L; d in {64, 96, 128, 256};
 *    L * d * 2 <= 2^32 (one head's Q, K or V within 4 GiB: L <= 2^23 at
 *    d = 256); B * H * L * d < 2^62.
 */
#ifndef PAPER_2609_10937_ATTN_H
#define PAPER_2609_10937_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ATTN_MAX_L (1 << 24)

typedef enum { ATTN_BF16 = 0, ATTN_F16 = 1, ATTN_F32 = 2 /* attn_gemm only */ } attn_dtype_t;

typedef enum {
  ATTN_OK = 0,
  ATTN_E_NULLPTR = -1,        /* a required pointer is NULL */
  ATTN_E_SHAPE = -2,          /* B, H or L outside the supported range */
  ATTN_E_UNSUPPORTED_D = -3,  /* head dimension not in {64, 96, 128, 256} */
  ATTN_E_DTYPE = -4,          /* dtype not an attn_dtype_t */
  ATTN_E_ALIGN = -5,          /* a tensor base address is not 16-byte aligned */
  ATTN_E_INFEASIBLE = -6,     /* tile derivation found no feasible tile (report.binding says why) */
  ATTN_E_NO_INSTANCE = -7,    /* derived tiles have no compiled kernel; never falls back */
  ATTN_E_HIP = -8,            /* a HIP runtime call failed */
  ATTN_E_WORKSPACE = -9,      /* workspace missing or smaller than required */
  ATTN_E_SCALE = -10,         /* scale is negative, NaN or infinite */
  ATTN_E_ARG = -11,           /* other invalid argument (descriptor field, preset name, atom id) */
  ATTN_E_DEVICE = -12,        /* the current device is not a usable gfx950 GPU */
  ATTN_E_SCRATCH = -13        /* attn_fwd_noalloc: split workspace above ATTN_NOALLOC_SCRATCH_BYTES */
} attn_status_t;

/* Size of the static per-GPU split workspace of attn_fwd_noalloc. */
#define ATTN_NOALLOC_SCRATCH_BYTES (32u << 20)

/* One matrix-core instruction shape (Section 3, MFMAAtom): D[m x n] += A[m x k] B[k x n],
 * inputs of in_bytes each, accumulation in acc_bytes. */
typedef struct {
  int32_t m, n, k;
  int32_t in_bytes, acc_bytes;
} attn_mfma_atom_t;

/* Hardware descriptor (Section 3, HardwareDescriptor): only the quantities the
 * derivation reads, plus peak figures used for reporting. */
typedef struct {
  int64_t lds_bytes;            /* LDS per CU (bytes) */
  int32_t vgpr_per_thread;      /* registers per lane at one wave per SIMD */
  int32_t wavefront_size;
  int32_t num_cus;
  int32_t simds_per_cu;
  int32_t lds_bytes_per_clk;    /* LDS read bandwidth per CU (0 = unknown) */
  int32_t mfma_flops_per_clk_cu;/* dense matrix-core flops per clock per CU (0 = unknown) */
  double hbm_tbps;              /* HBM bandwidth, TB/s */
  double peak_tflops;           /* dense matrix-core peak for the atom's input type */
  double clock_ghz;
  char name[32];
} attn_hw_desc_t;

/* The operation plus the fixed structure of the kernel family that will run it.
 * The structure fields are properties of a kernel design, chosen once; the
 * derivation never varies them. */
typedef struct {
  int32_t B, H, L, d;
  int32_t elem_bytes;           /* bytes per Q/K/V element */
  int32_t causal;
  int32_t kv_lds_num, kv_lds_den; /* share of LDS given to staged K/V tiles */
  int32_t kv_tiles;             /* t_KV x d tiles resident in that share */
  int32_t stage_tiles;          /* t_KV x d tiles staged through registers per step */
  int32_t score_tiles;          /* fp32 t_Q x t_KV score tiles live at once (2 when pipelined) */
  int32_t p_tiles;              /* t_Q x t_KV tiles of 16-bit weights held in registers for the
                                   second product (0 when they go through LDS, as in Section 6.1) */
  int32_t stat_regs;            /* registers per atom-row block of running statistics (the paper's
                                   (m, delta): 2) */
  int32_t operand_frags;        /* A-operand fragments of the atom in flight (read ahead of their
                                   products) */
  int32_t waves_per_wg;
  int32_t waves_per_simd;       /* resident waves per SIMD; divides the register file */
  int32_t vgpr_fixed;           /* registers per lane outside the counted arrays: lane addresses,
                                   copy offsets, constants (the paper's instance: 16) */
  int32_t max_split;            /* key-range splits the CU rule may use (1 = none) */
  int32_t wg_fixed_steps;       /* fixed cost of one workgroup (prologue, epilogue) in steps of one
                                   key tile, which the CU rule weighs against the tiles per split
                                   (0 = none) */
} attn_op_t;

/* Result of the derivation (Section 4: tiles, feasibility, binding constraint). */
typedef struct {
  int32_t feasible;
  int32_t t_kv;                 /* key/value rows per tile (fixed by LDS) */
  int32_t t_q_wave;             /* query rows per wave (fixed by registers) */
  int32_t n_waves;              /* waves per workgroup */
  int32_t tile_q;               /* query rows per workgroup = n_waves * t_q_wave */
  int32_t n_split;              /* key-range splits (1 = none); causal: the most pieces of one
                                   query tile's key range */
  int32_t tiles_per_split;      /* key tiles per split (causal: per piece of a query tile's own
                                   key range, the last piece of a tile holding the rest) */
  int64_t grid;                 /* workgroups launched by the fused kernel */
  int32_t vgpr_est, vgpr_budget;/* registers per lane at the GEMM1/GEMM2 sync point */
  int64_t lds_used, lds_budget;
  double wg_per_cu;
  int32_t low_occupancy;        /* grid < num_cus */
  int32_t lds_bw_ok;            /* t_q_wave * lds_bytes_per_clk >= mfma_flops_per_clk_cu */
  char binding[16];             /* "LDS", "VGPR", "CU" or "atom" */
  int64_t launch_grid;          /* workgroups the fused kernel is launched with: grid, or (from
                                   attn_fwd_plan) one per CU when attn_fwd runs the query tiles
                                   as a persistent launch, each workgroup taking a fixed list of
                                   them back to back (no split, more query tiles than CUs, each
                                   at least 4 and on average at most 24 key tiles long; d = 64
                                   and 128).  The derivation itself sets it to grid. */
} attn_tile_report_t;

/* Fill `out` with a named descriptor: "paper_gpu_a" and "paper_gpu_b" (the two
 * CDNA descriptors of Section 3), "gfx950" (MI355X public figures) or
 * "gfx942" (MI300X public figures; for the derivation only: the kernels are
 * built for gfx950).  ATTN_E_ARG for an unknown name. */
int attn_hw_desc_preset(const char* name, attn_hw_desc_t* out);

/* Descriptor of HIP device `device`: CU count, LDS size, wavefront size and
 * clock from the runtime, the rest from the gfx950 figures.  ATTN_E_DEVICE if
 * the device is not gfx950, ATTN_E_HIP if the runtime cannot be queried. */
int attn_hw_desc_query(int device, attn_hw_desc_t* out);

/* Named atoms: "f32_16x16x4" (the paper's), "bf16_16x16x32", "f16_16x16x32"
 * (gfx950), "bf16_16x16x16", "f16_16x16x16" (gfx942). */
int attn_atom_preset(const char* name, attn_mfma_atom_t* out);

/* Fill `out` with the operation (B, H, L, d, dtype, causal) and the structure
 * of this library's fused kernel family.  Same argument checks as attn_fwd. */
int attn_fwd_op(int B, int H, int L, int d, int causal, int dtype, attn_op_t* out);

/* Registers per lane live at the GEMM1/GEMM2 synchronisation point for a
 * given (t_q per wave, t_kv, waves per workgroup) -- the count behind Table 2. */
int attn_vgpr_estimate(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom,
                       const attn_op_t* op, int t_q_wave, int t_kv, int n_waves,
                       int32_t* out);

/* Closed-formula tile derivation (Sections 4 and 6.2): LDS fixes t_kv, the
 * register budget fixes t_q_wave, the CU count bounds the grid (splitting the
 * key range into the count with the fewest rounds of num_cus workgroups times
 * key tiles per split, then shrinking the Q tile if even the most splits leave
 * CUs idle), and every tile is atom aligned.
 * Returns ATTN_OK with report->feasible = 1, or ATTN_E_INFEASIBLE with
 * report->binding naming the constraint that failed.  Host-only integer math. */
int attn_tile_derive(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom,
                     const attn_op_t* op, attn_tile_report_t* report);

/* The report attn_fwd will act on for this shape: derivation over `hw`
 * (NULL = query the current device) plus the compiled-instance check
 * (ATTN_E_NO_INSTANCE if none matches). */
int attn_fwd_plan(const attn_hw_desc_t* hw, int B, int H, int L, int d, int causal, int dtype,
                  attn_tile_report_t* report);

/* Fused attention forward (Section 6: the attention equation, Algorithm 1 for
 * every Q tile, Figure 2's mapping).  scale: finite, >= 0 (1/sqrt(d) for
 * standard attention).  causal != 0 keeps keys j <= i for query i (top-left
 * aligned).  When the derivation splits the key range (split-N, Section 5.3),
 * a second kernel merges the splits' partial results with the Section 5.3
 * operator.  Plans whose report has launch_grid < grid run persistent: one
 * workgroup per CU, each taking its share of the query tiles back to back
 * (the result is the same, bit for bit).  The plan of each shape is derived
 * once per device and kept (at most 1024 shapes, then the table starts over).
 * Ownership and ordering: the call only enqueues work on `stream`; it never
 * synchronises.  The merge's workspace belongs to the library: one buffer per
 * (device, stream), so concurrent calls on different streams never share
 * one and calls on one stream use it in stream order.  A stream's buffer is
 * allocated (hipMalloc) on its first split call and grown when a larger shape
 * needs more; an outgrown buffer is kept, not freed, until process exit,
 * since work already enqueued may still use it.  Growing is refused while
 * `stream` is capturing (ATTN_E_WORKSPACE): capture after a call of the
 * same or a larger shape on that stream, or use attn_fwd_partial +
 * attn_fwd_merge with a caller-owned workspace, or attn_fwd_noalloc. */
int attn_fwd(const void* Q, const void* K, const void* V, void* O,
             int B, int H, int L, int d, float scale, int causal, int dtype, void* stream);

/* The two halves of attn_fwd, for callers that own the workspace (and for
 * timing the fused kernel on its own).  Split-N (Section 5.3): when the
 * derivation splits the key range, attn_fwd_partial runs the fused kernel
 * and leaves in `workspace`, per split and row, the split's output divided
 * by its own sum, rounded to the input type like O ([n_split][B*H][L][d],
 * 16-bit), followed by fp32 pairs ([n_split][B*H][L][2]) of the split's
 * reference point (scale*log2(e) times a logit at or below the row's
 * maximum; -inf for a row that saw none of the split's keys) and its sum;
 * attn_fwd_merge weighs the splits with the associative merge and writes O.
 * A causal plan (attn_fwd_plan) whose grid is below B*H * query tiles *
 * n_split has cut each query tile's own key tiles into pieces of
 * tiles_per_split and launches only the non-empty ones: slot k of a row is
 * then written only when the row's query tile has more than k pieces, and
 * attn_fwd_merge reads no other slot.
 * The normalised partials add one rounding to the input type before the
 * merge: |O - exact| <= 2u max|V| + fp32 terms (u = 2^-9 bf16, 2^-12 f16).
 * Without a split the required workspace is 0 bytes, attn_fwd_partial writes
 * O itself and attn_fwd_merge does nothing.  attn_fwd_workspace_bytes gives
 * the size for the current device; the workspace must be 16-byte aligned
 * (ATTN_E_WORKSPACE / ATTN_E_ALIGN otherwise).  attn_fwd_partial followed
 * by attn_fwd_merge on one stream equals attn_fwd bit for bit. */
int attn_fwd_workspace_bytes(int B, int H, int L, int d, int causal, int dtype, size_t* out);
int attn_fwd_partial(const void* Q, const void* K, const void* V, void* O,
                     int B, int H, int L, int d, float scale, int causal, int dtype,
                     void* workspace, size_t workspace_bytes, void* stream);
int attn_fwd_merge(const void* workspace, size_t workspace_bytes, void* O,
                   int B, int H, int L, int d, float scale, int causal, int dtype, void* stream);

/* attn_fwd for callers that cannot allocate device memory (code under stream
 * capture, serving loops, harnesses that forbid allocation): same arguments,
 * kernels and result as attn_fwd (bit for bit), with the split workspace in
 * a static array of ATTN_NOALLOC_SCRATCH_BYTES that each GPU holds from its
 * first call until process exit.  Never calls hipMalloc or hipFree.  A shape
 * whose split workspace (attn_fwd_workspace_bytes) exceeds the array is
 * refused with ATTN_E_SCRATCH before any device work.  All calls on one GPU
 * share the array: calls that overlap in time on that GPU (different streams,
 * concurrent graph replays) race and must be serialised by the caller. */
int attn_fwd_noalloc(const void* Q, const void* K, const void* V, void* O,
                     int B, int H, int L, int d, float scale, int causal, int dtype, void* stream);

/* Unfused baseline (Section 6.2, Table 3): three kernels on `stream` --
 * S = scale Q K^T written to the workspace in `dtype`, the row softmax of
 * attn_softmax overwriting S with P (masked entries 0), then O = P V.  The
 * two products run on the GEMM kernel of attn_gemm with the tiles
 * attn_gemm_derive gives for their shapes (L x L x d and L x d x L), in
 * fp32, written in `dtype`.  The workspace holds B*H*L*L elements; size it
 * with attn_unfused_workspace_bytes.  L must be a multiple of 8 and at most
 * 2^22 (ATTN_E_SHAPE otherwise). */
int attn_fwd_unfused(const void* Q, const void* K, const void* V, void* O,
                     int B, int H, int L, int d, float scale, int causal, int dtype,
                     void* workspace, size_t workspace_bytes, void* stream);
size_t attn_unfused_workspace_bytes(int B, int H, int L, int dtype);

/* Row softmax, the standalone online softmax of Section 5.3, on the same
 * CU-centric derivation.  A tile is one 16-byte load per lane of a wave
 * (wavefront_size * 16 / elem_bytes elements); the register budget (at the
 * kernel's 2 waves per SIMD, less its fixed registers) fixes how many tiles a
 * wave keeps resident, rounded down to a power of two; the CU rule splits a
 * row over up to the 4 waves of a workgroup (their running maximum and
 * denominator merged with the associative operator) until the grid reaches
 * the CU count.  A row segment that fits the resident tiles is read from HBM
 * once, else twice. */
typedef struct {
  int32_t feasible;
  int32_t tile_elems;       /* elements one wave moves per tile */
  int32_t resident_tiles;   /* tiles a wave keeps in registers */
  int32_t split;            /* waves sharing one row (1 = none) */
  int32_t waves_per_wg;
  int32_t rows_per_wg;
  int64_t seg;              /* row elements per wave (a multiple of 8) */
  int64_t grid;             /* workgroups launched */
  int32_t passes;           /* HBM reads of each element: 1 or 2 */
  int32_t vgpr_est, vgpr_budget;
  double wg_per_cu;
  int64_t hbm_bytes;        /* bytes read and written by one call */
  char binding[16];         /* "CU" (grid below the CU count), "VGPR" (two passes) or "none" */
} attn_softmax_report_t;

/* The derivation for a rows x n softmax of elem_bytes-byte elements.
 * Host-only integer math; ATTN_E_ARG for a bad descriptor, ATTN_E_SHAPE for
 * rows or n < 1. */
int attn_softmax_derive(const attn_hw_desc_t* hw, int64_t rows, int64_t n, int elem_bytes,
                        attn_softmax_report_t* out);

/* Y = softmax(X) along each row: y_ij = exp(x_ij - max_j x_ij) / sum_j exp(...),
 * X and Y [rows][n] contiguous in `dtype` (bf16 or f16), computed in fp32 and
 * rounded to nearest-even.  causal != 0 treats X as square n x n blocks stacked
 * along the rows and gives column j > (i mod n) of row i weight 0 (the
 * top-left mask of attention scores).  Y may equal X.  Pointers need 2-byte
 * alignment; with n % 8 == 0 and 16-byte aligned X and Y every access is a
 * 16-byte one.  rows >= 1, 1 <= n <= 2^31.  Asynchronous on `stream`. */
int attn_softmax(const void* X, void* Y, int64_t rows, int64_t n, int causal, int dtype, void* stream);

/* GEMM C = A B (Section 4's worked example, Figure 1): workgroup tile
 * t_M x t_N x t_K and per-wave tile from the same closed-form rules as the
 * attention tiles, for the fixed structure of the kernel family that runs the
 * atom (16-bit atoms: 5 LDS stages of an A and a B tile, 2 x 4 waves, 2 waves
 * per SIMD; 4-byte atoms: 3 stages, 2 x 2 waves, 1 wave per SIMD):
 *   LDS      t_M = t_N = floor(sqrt(LDS / elem)), aligned down to the atom
 *            times the waves along each side; t_K = floor(LDS / (stages
 *            (t_M + t_N) elem)), aligned down to the atom's k and to whole
 *            1 KB copy blocks per wave;
 *   VGPR     the per-wave accumulators, (t_M / W_M)(t_N / W_N) fp32 values
 *            over the wavefront, plus the fixed registers within the budget
 *            at the family's waves per SIMD (the larger side halves until
 *            they fit);
 *   CU count while ceil(M / t_M) ceil(N / t_N) is below the CU count the
 *            larger side halves, down to one atom per wave.
 * Section 4 prints the LDS rule with LDS / 2 under the square root; the
 * section's own numbers (128 x 128 x 32 for 64 KB, 4-byte elements, two
 * stages) follow from LDS / elem, which is the reading taken here. */
typedef struct {
  int32_t feasible;
  int32_t t_m, t_n, t_k;        /* workgroup (CU) tile */
  int32_t warp_m, warp_n;       /* per-wave tile of C */
  int32_t stages, waves_per_wg;
  int64_t grid;                 /* workgroups: ceil(M / t_m) ceil(N / t_n) */
  int32_t vgpr_est, vgpr_budget;
  int64_t lds_used, lds_budget;
  double wg_per_cu;
  char binding[16];             /* "LDS", "VGPR" or "CU" */
} attn_gemm_report_t;

/* The derivation for an M x N x K product with `atom` (its in_bytes is the
 * element size).  Host-only integer math; ATTN_E_ARG for a bad descriptor or
 * atom, ATTN_E_SHAPE for M, N or K < 1, ATTN_E_INFEASIBLE when not even one
 * atom per wave fits (report.binding says which resource). */
int attn_gemm_derive(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, int64_t M, int64_t N, int64_t K,
                     attn_gemm_report_t* out);

/* C = A B on the matrix cores: A [M][K] and B [K][N] row-major in `dtype`,
 * C [M][N] row-major fp32, every sum in fp32 (Section 5.1 validates the
 * GEMM against a double-precision reference).  bf16/f16 inputs run on the
 * 16x16x32 atom (products exact in fp32), fp32 inputs (ATTN_F32, the section's own
 * type) on the 16x16x4 fp32 atom, each with its kernel family's tiles from
 * attn_gemm_derive on the current device's descriptor.
 * Sizes: 1 <= M < 2^31; N and K multiples of 8 (bf16/f16) or 4 (fp32), at
 * least that, K <= 2^22 and N <= 2^24 (bf16/f16) or 2^22 (fp32)
 * (ATTN_E_SHAPE otherwise); A, B and C 16-byte aligned (ATTN_E_ALIGN).  C
 * must not overlap A or B.  Asynchronous on `stream`. */
int attn_gemm(const void* A, const void* B, float* C, int64_t M, int64_t N, int64_t K, int dtype, void* stream);

/* Matrix-core layout probe (Section 3.1: fragment ownership must be checked
 * on the hardware).  Runs one 16x16x32 product with atom 0 = bf16, 1 = f16:
 * A is a row-major 16 x 32 device array, Bm a row-major 32 x 16 array, C a
 * row-major 16 x 16 float array written through the fragment layouts the
 * attention kernel assumes.  C == A Bm iff those layouts are right. */
int attn_mfma_probe(int atom, const void* A, const void* Bm, float* C, void* stream);

const char* attn_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* PAPER_2609_10937_ATTN_H */
