/*
 * leech.h — C ABI of libleech: fused multi-shell Λ24(12) dequantize + GEMV
 * for AMD Instinct MI355X (gfx950).
 *
 * The library implements the batch-1 decode GEMV of "Unfolding the Leech
 * Lattice: Fused Multi-Shell Decoding and VRAM Layouts for 2-Bit LLM Weights":
 * weights are stored as 24-wide blocks, each the direction of a point of the
 * ball Λ24(12) (301 classes, 111,043,117,458,000 points, §2.1) times a scale.
 * An offline expansion turns each block's decoded fields (class id, gain bit,
 * sign mask, magnitude level per coordinate, §2.2) into one of four VRAM
 * layouts (§3.2); a HIP kernel reads a layout with shifts, masks and a table
 * lookup that is the same on every lane, and computes y = W x (§2.3).
 *
 * Conventions used by every call
 *   - Lattice points are integer vectors in the √8 scaling: shell m holds the
 *     points with Σ z_i² = 16 m; the ball is shells 2..12.
 *   - A class is a magnitude multiset.  Class ids follow the canonical order:
 *     ascending (shell m, even before odd, magnitudes sorted descending and
 *     compared lexicographically).  Ids 0..300; table slots 301..511 are zero.
 *   - The level of a coordinate is the index of |z_i| among the class's
 *     distinct magnitudes in ascending order (level 0 = smallest, 0 if the
 *     class has zero coordinates).  Bit i of a sign mask is 1 iff z_i < 0 and
 *     must be 0 where z_i = 0.
 *   - Weight of block b, coordinate i:
 *         w = scale_b · centroid[gain_b] · z_i / (4·√m_class)
 *     with scale_b an IEEE binary16 value and centroid[] two f32 values.
 *   - A matrix is M rows × Kpad columns, Kpad a multiple of 24, nb = Kpad/24
 *     blocks per row; block (r, j) covers columns 24j .. 24j+23 of row r.
 *     Host arrays of per-block fields are in row-major (r, j) order.
 *   - x is binary16 of length Kpad (zero-padded past the logical K); y is f32.
 *
 * Return values: LEECH_OK (0) or a negative LEECH_E_* code; the message of the
 * last failure on the calling thread is available from leech_last_error().
 * No call aborts or exits the process.
 *
 * Memory: the caller owns every buffer it passes and every stream.  Host
 * calls read and write host memory only.  Device calls take device pointers
 * (hipMalloc'd or equivalent), enqueue work on the given stream (a hipStream_t
 * passed as void*, NULL = the null stream) and return after enqueue; device
 * calls allocate no device memory.
 */
#ifndef LEECH_H
#define LEECH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
enum {
  LEECH_OK = 0,
  LEECH_E_ARG = -1,          /* null pointer or out-of-range scalar argument   */
  LEECH_E_LAYOUT = -2,       /* unknown layout kind                             */
  LEECH_E_SHAPE = -3,        /* M, Kpad or K not valid for the call             */
  LEECH_E_FIELD = -4,        /* a block's decoded fields are not valid          */
  LEECH_E_NOT_LATTICE = -5,  /* an integer vector is not a point of the ball    */
  LEECH_E_HIP = -6,          /* a HIP runtime call or kernel launch failed      */
  LEECH_E_CAPACITY = -7      /* an index field of the layout would overflow     */
};

/* Message describing the most recent failure on this thread ("" if none).
 * The pointer stays valid until the next library call on this thread. */
const char* leech_last_error(void);

/* ----------------------------------------------------------- codebook
 * The codebook of the ball Λ24(12) (§2.1, §2.3): the extended Golay code,
 * the 301 classes with their sizes, and the tables the kernels read.
 * Built on the host; immutable afterwards; safe to share between threads. */
typedef struct leech_codebook leech_codebook;

/* Build the codebook of the ball with shells 2..ball_m.  ball_m must be 12
 * (the ball the paper serves, §2.1) or 13 (the class-cardinality lock N(13)
 * of §2.4, for verification only; layouts and kernels need ball_m = 12). */
int leech_codebook_build(int ball_m, leech_codebook** out);
void leech_codebook_free(leech_codebook* cb);

/* n_classes: 301 for ball_m = 12.  n_points: the number of lattice points of
 * the ball, origin excluded (111043117458000).  index_bits: ceil(log2 N). */
int leech_codebook_info(const leech_codebook* cb, int* n_classes, uint64_t* n_points,
                        int* index_bits);

/* Per-class facts for class_id < n_classes: shell m, parity (0 even / 1 odd),
 * n_levels (1..5), levels[0..n_levels) = distinct magnitudes ascending,
 * size = number of lattice points in the class. */
int leech_codebook_class(const leech_codebook* cb, int class_id, int* shell, int* parity,
                         int* n_levels, uint8_t levels[5], uint64_t* size);

/* Tables held by the codebook, returned as a host pointer owned by the
 * codebook (valid until leech_codebook_free) and its size in bytes.  Device
 * calls take a device copy that the caller uploads.
 *   LEECH_TABLE_CLASS_LEVELS: 512 records of 24 bytes — five f32 level values
 *       a/(4√m) (round-to-nearest from f64) and a u32 level count, the class
 *       table of §2.3; slots past the last class are zero.
 *   LEECH_TABLE_CODEWORDS: 4096 u32, the extended Golay codewords sorted
 *       ascending (bit i = coordinate i).
 *   LEECH_TABLE_DEVICE: the table every GEMV/decode kernel reads: 512 records
 *       of 32 bytes (see LEECH_DEVICE_TABLE_BYTES); pass its device copy as
 *       d_class_table.
 *   LEECH_TABLE_GOLAY_GEN: 128 u32, the codewords of the 12-bit messages
 *       a (entries 0..63) and a << 6 (entries 64..127) under the code's
 *       generator; the codeword of message m is entry (m & 63) XOR entry
 *       64 + (m >> 6).  The Golay70 layout stores each block's codeword as its
 *       message; pass this table's device copy as d_codewords.
 *   LEECH_TABLE_INDEX: the format-v1 index table (class offsets and radices,
 *       the codewords by value and by weight, binomial coefficients), read by
 *       leech_transcode_planes14 as d_index_table; exists for the ball
 *       Λ24(12) and smaller balls (N < 2^47).
 * The per-class magnitudes and the Golay70 value tables are not tables of
 * their own: the magnitudes are in leech_codebook_class and in bytes 1..5 of
 * each LEECH_TABLE_DEVICE record, the Golay70 values in its bytes 16..31, so
 * the kernels read one 32-byte record per class. */
enum { LEECH_TABLE_CLASS_LEVELS = 0, LEECH_TABLE_CODEWORDS = 1, LEECH_TABLE_DEVICE = 2,
       LEECH_TABLE_INDEX = 3, LEECH_TABLE_GOLAY_GEN = 4 };
#define LEECH_TABLE_SLOTS 512
#define LEECH_DEVICE_TABLE_BYTES (512 * 32)
int leech_codebook_table(const leech_codebook* cb, int which, const void** host_ptr,
                         size_t* nbytes);

/* Decoded fields of n lattice points z (int8 [n][24], host).  Outputs (host,
 * caller-allocated): class_id[n], sign_mask[n], level[n][24].  Fails with
 * LEECH_E_NOT_LATTICE (first bad block index in the message) if a vector is
 * not a point of the ball. */
int leech_fields_from_points(const leech_codebook* cb, int64_t n, const int8_t* z,
                             uint16_t* class_id, uint32_t* sign_mask, uint8_t* level);

/* ------------------------------------------------------------ layouts
 * The four VRAM layouts of §3.2, all bit-exact (every block decodes to the
 * same integer point, class and gain bit):
 *   SLOT32     one-hot level masks (§3.2): class | gain | sign mask | one 24-bit
 *              mask per level above level 0; 16-byte records (≤ 4 levels) or
 *              20-byte records (5 levels); a side table locates each record.
 *   PLANES14   three binary bit planes and the sign plane (§2.2, §2.3) in a
 *              112-bit record at a uniform 14-byte stride; the served layout,
 *              4.80 b/w.  Bits (little-endian from the record's first byte):
 *              pair words W0 [0,32), W1 [32,64), W2 [64,96), class [96,105),
 *              gain 105, zero [106,112).  With c_i = p0|p1<<1|p2<<2 of
 *              coordinate i (its level + 1) and pos_i = 1 iff z_i ≥ 0, the
 *              96 plane bits are stored in the GPU's consumption order: the
 *              coordinates form 12 pairs (a_q, b_q) = (0,16), (4,20), (8,12),
 *              (1,17), (5,21), (9,13), (2,18), (6,22), (10,14), (3,19),
 *              (7,23), (11,15), and W_w rotated right by 4k and masked with
 *              0x08070807 is c_a | pos_a << 11 | c_b << 16 | pos_b << 27 for
 *              pair q = 4w + k (k = 0..3; the four rotations cover each bit
 *              of W_w once).
 *   PLANES12X  two bit planes and the sign plane in a 12-byte record for every
 *              block (§3.2, sub-4.3 b/w), in the GPU's consumption order: bits
 *              [0, 12) hold the block's table entry, class | gain << 9; the
 *              other bits hold, for each pair q of the PLANES14 pair list, its
 *              coordinates' 2-bit levels and non-negative bits at the places
 *              where one shift or rotation of the record's words leaves them in
 *              a byte-permute selector (the placement is part of the format and
 *              listed in the library's sources).  A block with five levels
 *              keeps its exact PLANES14 record in its tile's exception list,
 *              applied in the same launch; its record holds only the entry
 *              field, 1024 + its index in that list (at most 3072 exceptions a
 *              tile, LEECH_E_CAPACITY otherwise).  Exception entries are 16
 *              bytes: the record plus the block's slot in its tile in bits
 *              [106, 128).
 *   GOLAY70    9-byte record (§3.2, 3.6 b/w): bits [0, 12) the table entry
 *              (class | gain << 9), [12, 24) the 12-bit message of the block's
 *              codeword, [24, 48) and [48, 72) the low and high bits of a 2-bit
 *              in-class code per coordinate (bit i = coordinate i).  A block
 *              the 2-bit codes cannot hold is an exception as in PLANES12X:
 *              its record holds only the entry field, 1024 + its index in its
 *              tile's exception list.
 * PLANES12X and GOLAY70 keep their exception lists in side0 (the 16-byte
 * entries, tile after tile) and the index of each tile's first entry in side1
 * (a u32 per tile).
 * Records are stored in "wave tile" order: rows are grouped in tiles of
 * tile_rows rows; within a tile, each run of lane_cols consecutive blocks of
 * the tile's rows forms one unit of tile_rows · lane_cols ≤ 64 blocks, stored
 * row by row; a tile's units follow each other in column order.  The kernels
 * read one unit per wavefront step.  The geometry is part of the layout:
 * lane_cols is 1, 2, 3, 4, 8 or 16 and tile_rows a multiple of 4 with
 * tile_rows · lane_cols ≤ 64.  leech_expand_layout takes the library's choice
 * (leech_layout_geometry), which evens out the 256 CUs' work: with
 * L = ceil(tiles / 256) rounds of one tile per CU and a wave taking every 8th
 * unit of its tile, the choice has the least
 * L · 5 + max(L · units per wave, tiles · units per tile / 1792), plus for
 * three to six rounds 1.5 · (L − tiles / 256) · units per wave (the CUs a
 * partial last round leaves idle), ties going to more blocks per unit and
 * then to more tiles; where that choice is one round of 9 to 17 units per
 * wave, it moves to 257..512 tiles (two per CU, which a CU runs at once) of
 * at least 48 blocks per unit, at most ceil(units per wave / 2) + 1 units per
 * wave and no more rows per CU (the most blocks per unit, then the fewest
 * rows per CU, then the most tiles) (4096 × 4104: 4 × 16, i.e. lane_cols ×
 * tile_rows; 5120 × 5136: 3 × 20; 8192 × 8208: 2 × 32; 6144 × 4104 and
 * 8192 × 4104: 4 × 16; 34816 × 5136: 2 × 28;
 * 14336 × 4104: 1 × 64).  leech_expand_layout_tiled takes the caller's.
 */
enum { LEECH_SLOT32 = 0, LEECH_PLANES14 = 1, LEECH_PLANES12X = 2, LEECH_GOLAY70 = 3 };

typedef struct {
  int32_t layout;          /* LEECH_* layout kind                               */
  int32_t lane_cols;       /* blocks per row in one unit                        */
  int32_t tile_rows;       /* rows per tile (and per unit)                      */
  uint32_t tile_exc_max;   /* most exception blocks in one tile (PLANES12X,     */
                           /* GOLAY70; 0 for the other layouts)                 */
  int64_t M, Kpad, nb;     /* rows, padded columns, blocks per row              */
  uint64_t main_bytes;     /* bytes of the main record stream (incl. 16-B pad)  */
  uint64_t side_bytes[2];  /* side streams: exception table / per-tile offsets  */
  uint64_t n_exceptions;   /* blocks served from the exception table           */
  uint64_t served_bytes;   /* main + side streams + 2 B/block of fp16 scales   */
} leech_layout_desc;

/* Expand decoded fields into a layout (host, multithreaded).
 * Inputs (host, row-major (r, j)): class_id[M·nb], gain_bit[M·nb] (0/1),
 * sign_mask[M·nb], level[M·nb][24].  Every block is validated: class id in
 * range, level < the class's level count, no sign bit on a zero coordinate,
 * levels forming the class's magnitude multiset, no sign bits above bit 23;
 * the first bad block is named in the error.
 * Two-call protocol: with main_out == NULL only *desc is filled (sizes);
 * otherwise main_out/side0_out/side1_out must hold desc->main_bytes /
 * side_bytes[0] / side_bytes[1] bytes (a side pointer may be NULL when its
 * size is 0).  Fails with LEECH_E_SHAPE if Kpad % 24 != 0 or M, Kpad ≤ 0,
 * LEECH_E_LAYOUT for an unknown layout, LEECH_E_CAPACITY if a tile holds more
 * exceptions than its index field can name. */
int leech_expand_layout(const leech_codebook* cb, int layout, int64_t M, int64_t Kpad,
                        const uint16_t* class_id, const uint8_t* gain_bit,
                        const uint32_t* sign_mask, const uint8_t* level, void* main_out,
                        void* side0_out, void* side1_out, leech_layout_desc* desc);

/* leech_expand_layout with the caller's geometry: lane_cols in {1, 2, 3, 4,
 * 8, 16} and tile_rows a positive multiple of 4 with tile_rows · lane_cols ≤
 * 64 (LEECH_E_SHAPE otherwise); lane_cols = tile_rows = 0 takes the library's
 * choice, as leech_expand_layout does.  Every layout, kernel and entry point
 * serves every such geometry; the summation order of y depends on it. */
int leech_expand_layout_tiled(const leech_codebook* cb, int layout, int64_t M, int64_t Kpad,
                              int32_t lane_cols, int32_t tile_rows, const uint16_t* class_id,
                              const uint8_t* gain_bit, const uint32_t* sign_mask,
                              const uint8_t* level, void* main_out, void* side0_out,
                              void* side1_out, leech_layout_desc* desc);

/* The geometry leech_expand_layout picks for an M × Kpad matrix (the rule
 * above).  LEECH_E_SHAPE if M ≤ 0, Kpad ≤ 0 or Kpad % 24 != 0. */
int leech_layout_geometry(int64_t M, int64_t Kpad, int32_t* lane_cols, int32_t* tile_rows);

/* Permute per-block fp16 scales (host, row-major (r, j)) into the layout's
 * wave-tile order; scale_out holds M·nb binary16 values. */
int leech_layout_scales(const leech_layout_desc* desc, const uint16_t* scale_rowmajor,
                        uint16_t* scale_out);

/* Host-side decode of a layout (for verification): integer coordinates
 * z[M·nb][24], class_id[M·nb] and gain_bit[M·nb] in row-major (r, j) order.
 * Any output pointer may be NULL. */
int leech_host_decode_layout(const leech_codebook* cb, const leech_layout_desc* desc,
                             const void* main, const void* side0, const void* side1,
                             int8_t* z, uint16_t* class_id, uint8_t* gain_bit);

/* ------------------------------------------- format-v1 block codes (§2.1) */
/* A block code is a u64 holding the 47-bit direction index of a point of the
 * ball (bits 0..46) and the gain bit (bit 47); bits 48..63 are zero (2.000
 * bits per weight on disk).  The index enumerates the classes in id order,
 * then inside a class, as one mixed-radix number, most significant digit
 * first: even classes — the support codeword {i : |z_i| ≡ 2 mod 4} (rank
 * among the codewords of its weight, ascending value), the arrangement of the
 * support magnitudes, the arrangement of the other magnitudes, the signs of
 * the nonzero off-support coordinates, the signs of all support coordinates
 * but the last (whose sign the sum condition fixes); odd classes — the
 * codeword {i : z_i ≡ 3 mod 4} (rank among all 4096, ascending value) and the
 * arrangement of all 24 magnitudes (signs forced).  An arrangement is one
 * digit per level in ascending order: the colex rank of the level's positions
 * among those the smaller levels left free. */
#define LEECH_INDEX_BITS 47

/* Codes of n blocks given as decoded fields (host arrays, as for
 * leech_expand_layout) -> code[n] (host).  Multithreaded.  Every block is
 * validated as in leech_expand_layout; the first bad block is named in the
 * error (LEECH_E_FIELD, LEECH_E_NOT_LATTICE). */
int leech_index_encode(const leech_codebook* cb, int64_t n, const uint16_t* class_id,
                       const uint8_t* gain_bit, const uint32_t* sign_mask, const uint8_t* level,
                       uint64_t* code);

/* Decoded fields of n block codes (host, multithreaded): the load-time
 * transcoder's first half on the CPU (§2.2).  LEECH_E_FIELD names the first
 * code with bits above 47 set or an index ≥ N. */
int leech_index_decode(const leech_codebook* cb, int64_t n, const uint64_t* code,
                       uint16_t* class_id, uint8_t* gain_bit, uint32_t* sign_mask,
                       uint8_t* level);

/* The Planes14 descriptor of an M × Kpad matrix, without its fields (the
 * layout's size does not depend on the codes): what leech_expand_layout_tiled's
 * sizing call returns for LEECH_PLANES14 and this geometry (lane_cols =
 * tile_rows = 0: the library's choice). */
int leech_planes14_desc(int64_t M, int64_t Kpad, int32_t lane_cols, int32_t tile_rows,
                        leech_layout_desc* desc);

/* --------------------------------------------------------- device calls */

/* Fused dequantize + GEMV (§2.3): y[r] = Σ_j W[r][j] · x[j] with W decoded on
 * the fly from the layout.  d_main/d_side0/d_side1: the layout's streams;
 * d_class_table: device copy of LEECH_TABLE_DEVICE; d_codewords: device copy of
 * LEECH_TABLE_GOLAY_GEN (GOLAY70 only, else may be NULL); d_scale: fp16 scales
 * in wave-tile order (leech_layout_scales); centroid: the two f32 gain
 * centroids; d_x: binary16 [Kpad]; d_y: f32 [M].  Accumulates in f32; the
 * summation order depends only on (M, Kpad, lane_cols, tile_rows), so every
 * layout of one matrix in one geometry yields bit-identical y. */
int leech_gemv(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
               const void* d_side1, const void* d_class_table, const void* d_codewords,
               const uint16_t* d_scale, const float centroid[2], const uint16_t* d_x,
               float* d_y, void* stream);

/* Batched GEMV (§6 "Batching": one decode of each weight serves several
 * activations): Y[b] = W X[b] for b < batch, X[b] binary16 [Kpad] at
 * d_X + b·ldx, Y[b] f32 [M] at d_Y + b·ldy.  Each block is decoded once per
 * launch and multiplied with up to 16 activations staged in LDS; larger
 * batches run in chunks of 16 (fewer where Kpad leaves too little LDS: 16
 * activations fit up to about Kpad = 4,600, 8 up to about 9,200, the exact
 * bound depending on the column groups' rounding; where not even two fit,
 * the vectors run as single GEMVs).  Products as leech_set_batch_mode
 * selects: on the matrix cores (the default) Y[b][r] is within rounding of
 * leech_gemv on X[b] (tested within 2^-15 · Σ_j |W_rj · X[b]_j|), and a single
 * vector left after the 16-wide chunks still runs 2 wide; with v_dot2 Y[b]
 * is bit-identical to leech_gemv on X[b].  batch > 1 serves
 * LEECH_PLANES14 (LEECH_E_LAYOUT otherwise) and needs ldx ≥ Kpad, ldx a
 * multiple of 8 and ldy ≥ M (LEECH_E_ARG); batch = 1 is leech_gemv.  Other
 * arguments as leech_gemv. */
int leech_gemv_batch(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                     const void* d_side1, const void* d_class_table, const void* d_codewords,
                     const uint16_t* d_scale, const float centroid[2], int batch,
                     const uint16_t* d_X, int64_t ldx, float* d_Y, int64_t ldy, void* stream);

/* Row-grouped GEMV (§3.4: q/k/v and gate/up fused into row-concatenated
 * launches, each row with its own matrix's gain centroids): W is the row
 * concatenation of n_groups matrices sharing one activation, expanded as one
 * layout of M = Σ group_rows rows; group g's rows use the gain centroids
 * group_centroids[2g], group_centroids[2g + 1].  group_rows and
 * group_centroids are host arrays.  A tile may hold rows of two groups (each
 * lane then reads its own row's centroids), not of three: LEECH_E_SHAPE if a
 * tile holds two group boundaries other than at its first row, or if the rows
 * do not sum to M; LEECH_E_ARG for a non-finite centroid.  1 ≤ n_groups ≤
 * LEECH_MAX_GROUPS.  Other arguments as leech_gemv. */
#define LEECH_MAX_GROUPS 8
int leech_gemv_grouped(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                       const void* d_side1, const void* d_class_table, const void* d_codewords,
                       const uint16_t* d_scale, int n_groups, const int64_t* group_rows,
                       const float* group_centroids, const uint16_t* d_x, float* d_y,
                       void* stream);

/* How PLANES12X and GOLAY70 GEMVs enqueued from this call on (process-wide)
 * decode their exceptions, the blocks whose exact PLANES14 record sits in the
 * side list (§3.2: Golay70's plain decoder and one that hoists work out of
 * the per-slot path; Planes12x's correction of its five-level blocks).
 *   LEECH_EXC_HOISTED (default): each workgroup first decodes its tile's
 *     exception records densely and keeps each one's contribution in LDS as a
 *     table entry of its own; the per-block loop then runs the layout's own
 *     decode alone, and an exception lane's lookup yields its kept value.
 *   LEECH_EXC_INLINE: every wave step that holds an exception decodes it in
 *     the loop, beside the layout's decode of the other lanes.
 * Both give bit-identical y.  A tile whose exception records exceed the LDS
 * budget is decoded in line either way.  LEECH_E_ARG for another value. */
enum { LEECH_EXC_HOISTED = 0, LEECH_EXC_INLINE = 1 };
int leech_set_exception_mode(int mode);

/* Products of leech_gemv_batch calls with batch > 1 enqueued from this call on
 * (process-wide; §6 "Batching").  LEECH_BATCH_AUTO (default): each decoded
 * block meets its activations on the matrix cores (16-block 4×4×4 binary16
 * products with f32 accumulation, one block's 24 products per output, so the
 * block's scale and class factor still multiply its f32 dot product); Y[b] is
 * then within rounding of leech_gemv on X[b] (the matrix core sums a block's
 * products in its own order) and bit-identical for a given X[b] whatever the
 * batch size or X[b]'s position.  LEECH_BATCH_DOT2: v_dot2 per activation,
 * Y[b] bit-identical to leech_gemv on X[b].  LEECH_E_ARG for another value. */
enum { LEECH_BATCH_AUTO = 0, LEECH_BATCH_DOT2 = 1 };
int leech_set_batch_mode(int mode);

/* Order in which single (non-batched, non-rotated) GEMVs enqueued from this
 * call on (process-wide) request their weight records, for measurement (§2.3:
 * the kernel streams the records; §3.4 attributes the gap to the DRAM floor
 * largely to latency and occupancy).  Every wave keeps 8 (mode 2: 6) units
 * (tile_rows × lane_cols blocks each) in flight; before the workgroup's staging barrier it requests
 * all 8 (mode 0), 3 (mode 1) or 2 (mode 2) of them, and the rest one per step
 * afterwards.  LEECH_PROLOGUE_AUTO (default) picks by the units a wave
 * streams: ≤ 6 -> 2, ≤ 16 -> 1, more -> 0.  The summation order does not
 * depend on the mode: y is bit-identical in every mode.  LEECH_E_ARG for
 * another value. */
enum { LEECH_PROLOGUE_AUTO = -1 };
int leech_set_prologue_mode(int mode);

/* Measurement launch: leech_gemv (PLANES14 only; LEECH_E_LAYOUT otherwise)
 * that also records, per workgroup t, 11 u64 stamps of the GPU's 100 MHz
 * real-time counter at d_stamps[11·t + k] (caller-owned device memory, 8-byte
 * aligned, 11 · ceil(M / tile_rows) entries): k = 0 the first wave's start,
 * 1 the first wave past the staging barrier (x and the class table in LDS),
 * 2 + w wave w's last unit decoded (w < the launch's waves; the rest are not
 * written), 10 the first wave's last y store issued.  The work and y are
 * leech_gemv's; the stamps cost one counter read and one store each.  For the
 * phase breakdown of a launch (§3.4 attributes the gap to the DRAM floor to
 * latency, occupancy and staging). */
int leech_gemv_phases(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                      const void* d_side1, const void* d_class_table, const void* d_codewords,
                      const uint16_t* d_scale, const float centroid[2], const uint16_t* d_x,
                      float* d_y, uint64_t* d_stamps, void* stream);

/* GEMV behind the activation rotation in one launch (§2.3: the activation is
 * rotated before the matvec; §6: every consumer rotates): y = W · R(x), where
 * R is leech_rotate_x's blockwise Walsh–Hadamard rotation of the raw binary16
 * activation d_x [K] with the signs d_signs [K] (NULL: all +1).  Each
 * workgroup rotates the activation in LDS while its first weight loads are in
 * flight; the result is bit-identical to leech_rotate_x(K, Kpad, d_x,
 * d_signs, xr) followed by leech_gemv_grouped(…, xr, d_y).  Row groups and
 * centroids as leech_gemv_grouped (n_groups = 1 for a plain GEMV).  Serves
 * LEECH_PLANES14 (LEECH_E_LAYOUT otherwise); needs 0 < K ≤ Kpad, K a multiple
 * of 8, the power-of-two factor of K at most 32768, K at most 40 × the
 * workgroup's threads (20480 for matrices of 512 or more rows) and the
 * rotation buffer within LDS (LEECH_E_SHAPE otherwise); d_x 16-byte and
 * d_signs 8-byte aligned. */
int leech_gemv_rotated(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                       const void* d_side1, const void* d_class_table, const void* d_codewords,
                       const uint16_t* d_scale, int n_groups, const int64_t* group_rows,
                       const float* group_centroids, int64_t K, const uint16_t* d_x,
                       const int8_t* d_signs, float* d_y, void* stream);

/* Verification decode on the device with the GEMV's own decoders (§2.4
 * "Verification": every block of a served matrix decoded and compared bit for
 * bit with the reference decode): z int8 [M·nb][24], class_id [M·nb],
 * gain_bit [M·nb], row-major (r, j).  Any output may be NULL.  LEECH_E_SHAPE
 * for a descriptor that is not valid, LEECH_E_ARG for a missing stream or
 * table or a misaligned pointer (d_z and d_main 4-byte, d_side1 8-byte),
 * LEECH_E_LAYOUT for an unknown layout, LEECH_E_HIP if the launch fails. */
int leech_decode_blocks(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                        const void* d_side1, const void* d_class_table,
                        const void* d_codewords, int8_t* d_z, uint16_t* d_class_id,
                        uint8_t* d_gain_bit, void* stream);

/* FP16 GEMV control (§3.2, Table "layout scale" first row): y = W x with W a
 * row-major binary16 [M][K] matrix, f32 accumulation.  K must be a multiple of
 * 8 and d_W 16-byte aligned. */
int leech_fp16_gemv_ref(int64_t M, int64_t K, const uint16_t* d_W, const uint16_t* d_x,
                        float* d_y, void* stream);

/* No-weights control (§3.3 "The no-weights control"): the GEMV's launch
 * geometry, x staging and reductions for this layout's shape, reading no
 * weight bytes: every block is taken as all-ones with unit scale, so
 * y[r] = Σ_j x[j] (f32, the GEMV's summation order). */
int leech_noweights_ctrl(const leech_layout_desc* desc, const uint16_t* d_x, float* d_y,
                         void* stream);

/* Activation rotation (§2.3 "The kernel", §6 "The rotated basis"): weights
 * live in a rotated basis, so the activation is rotated before the GEMV.  For
 * K = n·m with n = 2^k the largest power of two dividing K (n ≤ 32768), every
 * block b of n consecutive coordinates becomes
 *     xr[b·n + i] = n^(-1/2) · Σ_j H_n[i][j] · s[b·n + j] · x[b·n + j],
 * H_n[i][j] = (−1)^popcount(i & j) (Sylvester-ordered Walsh–Hadamard), with s
 * the caller's signs (int8 [K]: a negative entry means −1, any other +1;
 * NULL = all +1).  d_x: binary16 [K]; d_xr: binary16 [Kpad], the f32 result
 * rounded to nearest even, zero past K, ready as the GEMV's activation;
 * d_xr32: optional f32 [K] copy of the values before that rounding (NULL to
 * skip).  All pointers are caller-owned device memory; d_x and d_xr need
 * 2-byte, d_xr32 4-byte alignment (16-byte alignment of every pointer, and
 * 8-byte of d_signs, lets the kernel use vector loads and stores).
 * Arithmetic in f32; asynchronous on `stream`.  LEECH_E_ARG for a NULL d_x or
 * d_xr or a misaligned pointer; LEECH_E_SHAPE if K ≤ 0, Kpad < K or
 * n > 32768. */
int leech_rotate_x(int64_t K, int64_t Kpad, const uint16_t* d_x, const int8_t* d_signs,
                   uint16_t* d_xr, float* d_xr32, void* stream);

/* Load-time transcoder on the device (§2.2: each block's index is expanded
 * once into its decoded-field record): format-v1 codes -> the Planes14 main
 * stream, bit-identical to leech_expand_layout's.  desc: a Planes14
 * descriptor (leech_planes14_desc); d_index_table: device copy of
 * LEECH_TABLE_INDEX; d_code: u64 [M·nb], row-major (r, j); d_main:
 * desc->main_bytes bytes, every one written (trailing pad included);
 * d_bad: one u32 on the device, set to the number of codes that are not
 * format-v1 codes (their records are written as zeros; the caller must treat
 * the stream as invalid when it is nonzero).  Asynchronous on `stream`.
 * Alignment: d_main and d_index_table 16 bytes, d_code 8 (LEECH_E_ARG
 * otherwise).  LEECH_E_LAYOUT if desc is not Planes14. */
int leech_transcode_planes14(const leech_layout_desc* desc, const void* d_index_table,
                             const uint64_t* d_code, void* d_main, uint32_t* d_bad,
                             void* stream);

#ifdef __cplusplus
}
#endif
#endif /* LEECH_H */
