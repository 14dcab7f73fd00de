/*
 * lego.h - C ABI of the MI355X (gfx950) layout-mapped data-movement library.
 *
 * Implements the layout algebra of "LEGO: A Layout Expression Language for Code
 * Generation of Hierarchical Mapping" (Tavakkoli, Oancea, Hall; arXiv
 * 2505.08091): bijective hierarchical layouts built from tile shapes, constant
 * permutations of dimensions (RegP) and user-level irregular permutations
 * (GenP), chained by OrderBy under a GroupBy logical view (Section III-B,
 * Figures 3-5).  Layouts are lowered to straight-line integer index code
 * (Section IV-A) that is compiled at run time for gfx950 into three kinds of
 * kernel: index-map evaluation, layout remap, and a tiled MFMA GEMM whose
 * operand, LDS, fragment and workgroup-schedule layouts are layouts.
 *
 * Conventions
 *  - Every function returns lego_status; LEGO_OK (0) on success, a negative
 *    code on failure, and never aborts.  lego_last_error() returns a
 *    thread-local message for the last failure on the calling thread.
 *  - Indices and sizes are int64_t.  Tile dimension arrays are row-major lists
 *    of positive sizes.  Permutations (sigma) are 1-based, as in the paper, and
 *    act as gathers: sigma(v)_k = v[sigma_k].
 *  - Handles (lego_piece_t, lego_layout_t) are created by the library,
 *    immutable and reference counted.  Composition retains its inputs, so a
 *    caller may release a piece as soon as it has been composed.  Release every
 *    handle it created with lego_release().
 *  - Device entry points are asynchronous on the caller's stream (a
 *    hipStream_t passed as void*, NULL = the null stream).  All device memory is
 *    owned by the caller; the library never frees it and allocates no device
 *    memory.  The first call with a new layout combination compiles a kernel
 *    (hipRTC, cached in memory and on disk); later calls only launch.  Launch
 *    errors are returned; faults inside a kernel surface at the caller's next
 *    synchronisation.
 */
#ifndef LEGO_H
#define LEGO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int lego_status;
enum {
  LEGO_OK = 0,
  LEGO_E_INVALID_ARG = -1,    /* null pointer, bad rank, non-positive size, bad kind */
  LEGO_E_SIZE_MISMATCH = -2,  /* element counts of GroupBy and an OrderBy differ (Section III-B, correctness) */
  LEGO_E_NOT_PERMUTATION = -3,/* sigma is not a permutation of [1..d] */
  LEGO_E_OUT_OF_RANGE = -4,   /* an index outside the layout's space */
  LEGO_E_NOT_BIJECTIVE = -5,  /* brute-force check found a collision or a gap */
  LEGO_E_UNSUPPORTED = -6,    /* valid request the library does not implement */
  LEGO_E_JIT = -7,            /* run-time compilation of a generated kernel failed */
  LEGO_E_HIP = -8,            /* a HIP runtime call failed */
  LEGO_E_NO_MEMORY = -9
};

/* Message for the last failure on this thread ("" if none). */
const char* lego_last_error(void);
/* Library version string. */
const char* lego_version(void);

typedef struct lego_piece_s* lego_piece_t;   /* a RegP or GenP permutation of one tile */
typedef struct lego_layout_s* lego_layout_t; /* a GroupBy chain (or ExpandBy) */

/* Handles are reference counted: a new handle holds one reference,
 * lego_retain adds one, lego_release drops one and frees the handle with the
 * last.  Composition keeps what it needs, so a piece may be released right
 * after it has been composed into a layout.  NULL is ignored by both. */
void lego_retain(void* handle);
void lego_release(void* handle);

/* ---------------------------------------------------------------- pieces --
 * RegP(tile, sigma) (Figure 3; apply/inv in Figure 4): a constant permutation
 * of the dimensions of a d-dimensional tile.  dims[d] > 0, sigma[d] 1-based.
 * Errors: INVALID_ARG (d < 1, d > 16, null pointer, size <= 0),
 * NOT_PERMUTATION. */
lego_status lego_regp(int d, const int64_t* dims, const int32_t* sigma, lego_piece_t* out);

/* Row([n1..nd]) = RegP(n, [1..d]): row-major (sugar after Equation (2)). */
lego_status lego_row(int d, const int64_t* dims, lego_piece_t* out);

/* Col([n1..nd]) = RegP([n1..nd], [d..1]): column-major with the logical dims
 * kept in order, first index fastest (the meaning the paper uses for column-
 * major operands in Section V-A). */
lego_status lego_col(int d, const int64_t* dims, lego_piece_t* out);

/* GenP(tile, f, f^-1) (Figure 3; Figure 4): an irregular bijection of the tile's
 * elements, from a fixed catalogue (user functions cannot cross a C ABI that
 * must also lower them to kernel code):
 *   LEGO_GENP_MORTON      2D, power-of-two sides; Z order (column bits at even
 *                         positions), no params.
 *   LEGO_GENP_XOR_SWIZZLE 2D [R,C]; params {v, s}: vectors of v elements of row
 *                         r are XOR-permuted by (r/s) mod (C/v); C/v a power of two.
 *   LEGO_GENP_REVERSE     any rank; every coordinate reversed (Figure 2's p).
 *   LEGO_GENP_ANTIDIAG    2D square; antidiagonal order of Figure 7.
 * Errors: INVALID_ARG (bad kind, shape or params). */
enum { LEGO_GENP_MORTON = 1, LEGO_GENP_XOR_SWIZZLE = 2, LEGO_GENP_REVERSE = 3, LEGO_GENP_ANTIDIAG = 4 };
lego_status lego_genp(int kind, int d, const int64_t* dims, const int64_t* params, int nparams,
                      lego_piece_t* out);

/* A user-defined GenP (Section III-B: any bijection f with its inverse) given
 * as integer expressions, so that it evaluates on the host and lowers to
 * kernel code like the built-in GenPs (the paper writes f in Python; text is
 * what crosses a C ABI).  apply_expr: the physical index within the tile as a
 * function of the coordinates i0..i{d-1} (i, j, k alias the first three);
 * inv_exprs: d expressions separated by ';', coordinate k as a function of x.
 * Both may use the tile extents n0..n{d-1}.  Language: integers, + - * and
 * floor / % by positive constants, << >> by constants, & with a constant mask
 * 2^k - 1, ^ on non-negative values, < <= > >= == != ! && || (C truth
 * values, results 0/1), c ? a : b, parentheses, isqrt (exact floor square root), min, max;
 * C precedence.  The forward result is taken modulo the tile size and inverse
 * coordinate k modulo n_k (the identity for a bijection, and a range the
 * lowering can use).  Tiles of at most 2^20 points are checked exhaustively on
 * construction (NOT_BIJECTIVE when f is not a bijection onto [0, size) or the
 * inverse does not undo it); larger ones can be checked with
 * lego_verify_bijective.  Errors: INVALID_ARG (syntax, unsupported operation,
 * with the offset in lego_last_error), NOT_BIJECTIVE. */
lego_status lego_genp_expr(int d, const int64_t* dims, const char* apply_expr, const char* inv_exprs,
                           lego_piece_t* out);

/* Rank and dims of a piece; dims must hold 16 entries. */
lego_status lego_piece_dims(lego_piece_t p, int* rank, int64_t* dims);

/* --------------------------------------------------------------- layouts --
 * GroupBy(tiles) (Figure 3; Figure 5): the logical view.  dims is the
 * concatenation of the tile levels; the logical index has rank entries.
 * Errors: INVALID_ARG. */
lego_status lego_groupby(int rank, const int64_t* dims, lego_layout_t* out);

/* GroupBy(T^1..T^q) over q tile levels of d dimensions each (Figure 3's
 * grammar names the levels): tiles[q*d], level-major.  The logical index is
 * the concatenation of the levels' coordinates (q*d entries), so this is
 * lego_groupby(q*d, tiles) with the level structure checked.  Errors:
 * INVALID_ARG (q < 1, d < 1, q*d > 64, null, size <= 0). */
lego_status lego_groupby_tiles(int q, int d, const int64_t* tiles, lego_layout_t* out);

/* base.OrderBy(P_1..P_n) (Equation (2) dot notation): appends a reordering; the
 * chain is applied in call order by apply.  Errors: INVALID_ARG,
 * SIZE_MISMATCH (element counts differ). */
lego_status lego_orderby(lego_layout_t base, int n, const lego_piece_t* pieces, lego_layout_t* out);

/* TileBy_{q x d}(T^1..T^q) (sugar after Equation (2)): tiles[q*d] tile sizes,
 * level-major.  Logical index = tile coordinates of every level; apply gives
 * the row-major position in the full tensor. */
lego_status lego_tileby(int q, int d, const int64_t* tiles, lego_layout_t* out);

/* TileOrderBy_{q x d}(P^1..P^q): logical index = full coordinates (extents
 * N_k = prod_h n^h_k); apply gives the position in tile-major storage whose
 * level h is ordered by piece P^h, each of rank d.  (The printed definition is
 * garbled; this is the reading that maps full coordinates to hierarchically
 * tiled storage.)  Errors: INVALID_ARG (q < 1, null, a level not of rank d). */
lego_status lego_tileorderby(int q, int d, const lego_piece_t* levels, lego_layout_t* out);

/* GroupBy(P.dims).OrderBy(P): a single permutation used as a whole layout. */
lego_status lego_layout_from_piece(lego_piece_t p, lego_layout_t* out);

/* ExpandBy(n, n', G) (Figure 9, Section III-D): partial tiles.  G is a layout
 * over the padded extents n' (prod n' = size of G); apply returns -1 for logical
 * points outside n.  Host evaluation and index-map kernels only. */
lego_status lego_expandby(int d, const int64_t* n, const int64_t* n_expanded, lego_layout_t g,
                          lego_layout_t* out);

/* Queries.  dims must hold `cap` entries (rank <= 64). */
lego_status lego_layout_rank(lego_layout_t l, int* rank);
lego_status lego_layout_dims(lego_layout_t l, int cap, int64_t* dims);
lego_status lego_layout_size(lego_layout_t l, int64_t* n); /* logical points */
/* Physical positions: the original extents' product for an ExpandBy layout
 * (Figure 9), the logical size otherwise.  A buffer in this layout holds this
 * many elements. */
lego_status lego_layout_phys_size(lego_layout_t l, int64_t* n);

/* Host evaluation (Figures 4-5).  apply: idx[rank] logical -> *flat physical.
 * inv: physical flat -> idx[rank].  Errors: OUT_OF_RANGE. */
lego_status lego_apply(lego_layout_t l, const int64_t* idx, int64_t* flat);
lego_status lego_inv(lego_layout_t l, int64_t flat, int64_t* idx);

/* Opt-in brute-force bijection check over all points (the first correctness
 * condition is the user's duty; this verifies it).  Refuses layouts with more
 * than max_points points (INVALID_ARG).  Returns NOT_BIJECTIVE on failure. */
lego_status lego_verify_bijective(lego_layout_t l, int64_t max_points);

/* The lowered index code of apply (which = 0, as a function of the logical flat
 * index x) or inv (which = 1, of the physical index p), as HIP/C++ text, with
 * the operation counts of both lowering variants in a comment (the analogue of
 * Table IV).  Writes at most cap bytes including the NUL; *need receives the
 * full length + 1. */
lego_status lego_emit(lego_layout_t l, int which, char* buf, size_t cap, size_t* need);

/* ---------------------------------------------------------------- device --
 * Index maps on the GPU (bit-exact with host evaluation).
 * apply_all: d_out[x] = apply(B^{-1}(x)) for every logical flat x, idx_bytes
 *   = 4 (int32) or 8 (int64); d_out holds size elements.
 * inv_all: d_out[p*rank + k] = inv(p)[k] for every physical p.
 * d_out must be 16-byte aligned (the kernels store 16-byte vectors).
 * Errors: INVALID_ARG, JIT, HIP. */
lego_status lego_apply_all_device(lego_layout_t l, int idx_bytes, void* d_out, void* stream);
lego_status lego_inv_all_device(lego_layout_t l, int idx_bytes, void* d_out, void* stream);

/* Remap: for every logical x, the element at src.apply(x) of d_src moves to
 * dst.apply(x) of d_dst (elem_bytes = 1, 2, 4 or 8; the copy is bit-exact).
 * The layouts must have equal logical dims.  d_src holds src's physical size
 * in elements and d_dst dst's (they differ from the logical size only for
 * ExpandBy layouts, Section III-D / Figure 9).  With an ExpandBy source, a
 * destination position whose logical point lies outside the source's original
 * extents (src.apply = -1) receives zero (padding); with an ExpandBy
 * destination, logical points outside its extents are not copied (cropping).
 * d_src and d_dst must not overlap and must be 16-byte aligned.  Errors:
 * INVALID_ARG, SIZE_MISMATCH, UNSUPPORTED, JIT, HIP. */
lego_status lego_remap(lego_layout_t src, lego_layout_t dst, int elem_bytes, const void* d_src, void* d_dst,
                       void* stream);

/* The plan lego_remap would use: path 0 direct vector copy, 1 LDS-tiled, 2
 * element gather, 3 box-staged (a 2-D map without digit structure, such as
 * the antidiagonal order of Figure 7, copied through LDS one square box of
 * the logical index space at a time, read and written in the orders under
 * which each side is contiguous); run = contiguous run length of the map;
 * vec = elements per vector; tile = elements per LDS tile or box (0 if none).  info (may be NULL) gets a
 * text summary of at most info_cap bytes. */
lego_status lego_remap_plan(lego_layout_t src, lego_layout_t dst, int elem_bytes, int* path, int64_t* run,
                            int* vec, int64_t* tile, char* info, size_t info_cap);

/* GEMM C = A * B (Section II and V-A): fp16 or bf16 inputs, fp32 accumulation
 * on the gfx950 matrix cores, fp32 C.  Every index is a layout:
 *   a     over [M,K]  (NULL: Row(M,K))      b over [K,N] (NULL: Col(K,N))
 *   c     over [M,N]  (NULL: Row(M,N))
 *   sched over [M/bm, N/bn]: tile (tm,tn) is computed by workgroup
 *         sched.apply(tm,tn) (NULL: group_m-grouped order, column-major inside
 *         a group, the order the paper's Triton matmul uses)
 *   lds_a over [bm, bk] and lds_b over [bn, bk]: element offsets in the LDS tile
 *         (NULL: XOR swizzle GenP with 16-byte vectors)
 * frag_a, frag_b, frag_c: the register fragment layouts of the MFMA
 *         instruction, as lego_mfma_fragment_layout returns them (logical
 *         (lane, element) -> position in the A, B or C block).  The hardware
 *         fixes them per instruction, so given layouts select the instruction
 *         (32x32x16 or 16x16x32) whose fragments they are, compared point by
 *         point; layouts of no instruction, or of different ones, are
 *         UNSUPPORTED.  NULL: 32x32x16 when the wave tile allows it.  xcd_remap != 0 composes a layout that keeps
 * consecutive tiles of the schedule on one XCD.  M, N and K need not be
 * multiples of the tile (partial tiles, Section III-D): the tile counts round
 * up, operand elements outside [M,K] / [K,N] load as zero and C elements
 * outside [M,N] are not stored; operand layouts are plain (an ExpandBy
 * operand is UNSUPPORTED).  d_a and d_b must be 16-byte aligned, d_c 4-byte
 * aligned, and C must not overlap A or B (INVALID_ARG).  Errors: INVALID_ARG,
 * SIZE_MISMATCH, UNSUPPORTED, JIT, HIP. */
enum { LEGO_F32 = 0, LEGO_F16 = 1, LEGO_BF16 = 2 };
typedef struct {
  int64_t M, N, K;
  int in_dtype;          /* LEGO_F16 or LEGO_BF16 */
  int bm, bn, bk;        /* workgroup tile; 0 = default 256x256x64 */
  int wm, wn;            /* wave tile; 0 = default (bm/2, bn/2) */
  int group_m;           /* grouping of the default schedule; 0 = 8 */
  int xcd_remap;         /* 1 = keep consecutive scheduled tiles on one XCD */
  int stages;            /* LDS stages of the k loop (2..4, within 160 KiB of LDS);
                            0 = chosen; a count the plan cannot use is UNSUPPORTED */
  int max_workgroups;    /* plans whose workgroups walk several tiles (the plan
                            text says "persistent"): launch at most this many
                            workgroups; 0 = as many as the device holds at once */
  lego_layout_t a, b, c, sched, lds_a, lds_b;
  lego_layout_t frag_a, frag_b, frag_c;  /* MFMA fragment layouts (see below); NULL: chosen */
} lego_gemm_desc;
lego_status lego_gemm(const lego_gemm_desc* desc, const void* d_a, const void* d_b, float* d_c, void* stream);

/* Text summary of the GEMM plan (tile, waves, vector paths, op counts). */
lego_status lego_gemm_plan(const lego_gemm_desc* desc, char* info, size_t info_cap);

/* The MFMA fragment layout of operand (0 = A, 1 = B, 2 = C/D) of instruction
 * (0 = v_mfma_f32_32x32x16 f16/bf16, 1 = v_mfma_f32_16x16x32 f16/bf16) as a
 * layout: logical (lane, element) -> physical row*cols + col within the block. */
lego_status lego_mfma_fragment_layout(int instr, int operand, lego_layout_t* out);

/* Compile every generated kernel source for the built-in test and benchmark
 * configurations with hipRTC (no GPU needed).  Returns the number of sources
 * compiled in *count; info (may be NULL) gets a first line naming the
 * compiler ("compiler: hipRTC <major>.<minor> from <library>"), then one
 * line per source with its compile time.  Used by the build check.
 *
 * Kernels are compiled by the hipRTC of the installed ROCm (ROCM_PATH,
 * default /opt/rocm), loaded into a link namespace of its own so that a
 * host process carrying another ROCm release's compiler library does not
 * substitute it.  LEGO_DUMP=<dir> keeps each generated source and its code
 * object there. */
lego_status lego_selftest_compile(int* count, char* info, size_t info_cap);

/* The generated kernel source a device call would compile (for inspection and
 * host-side verification of the lowered index code): kind 0 = apply_all and
 * 1 = inv_all of layout a with param = idx_bytes; 2 = remap from a to b with
 * param = elem_bytes; 3 = GEMM described by desc.  Text as in lego_emit. */
lego_status lego_plan_source(int kind, lego_layout_t a, lego_layout_t b, int param, const lego_gemm_desc* desc,
                             char* buf, size_t cap, size_t* need);

/* The index-th generated source of the built-in configurations (its name and
 * full text), for host-side inspection and verification of the lowered index
 * code.  Returns OUT_OF_RANGE past the last one; *need = text length + 1. */
lego_status lego_selftest_source(int index, char* name, size_t name_cap, char* src, size_t src_cap, size_t* need);

#ifdef __cplusplus
}
#endif

#endif /* LEGO_H */
