/*
 * wc.h -- C ABI of libwc, the MI355X chunked rANS weight decoder.
 *
 * The library turns near-entropy-bound compressed weight streams back into
 * bit-identical bf16 / fp16 / int8 / int4 / fp8 / fp4 tensors in GPU memory
 * (wc_decode), or multiplies weights into activations while decoding them,
 * never writing them out (wc_gemv, wc_gemm: bf16 and fp8; wc_gemm_i8: int8;
 * wc_gemv_mx: MXFP4; wc_gemv_w4: int4 with group scales).  Compression runs on the host (wc_encode) or on the GPU
 * (wc_encode_device), to the same blob.
 *
 * Paper: "Approaching Shannon Bound with Lossless LLM Weight Compression"
 * (Tan, Chen, Alonso, Wong, He).
 *   - Sec. II-B: per-tensor empirical entropy over format-defined symbols.
 *   - Sec. IV-A, V-B: weights cut into independently decodable ANS
 *     substreams with a static frequency table and an offset index; the
 *     compression is offline.
 *   - Alg. 2, Sec. V-C-3: lane-parallel rANS decode with a table lookup of
 *     (symbol, frequency, cumulative frequency) in on-chip memory and
 *     coalesced renormalisation reads.
 *   - Alg. 1 / 3, Sec. V (pipeline overlap and the batch-size regime):
 *     decoded tiles consumed by the GEMM on chip, never written to memory.
 *   - Sec. VI-F: metadata = 4 B per tile offset + one 2^12-entry codebook.
 *
 * All functions return a wc_status; no C++ exception crosses the ABI.  No
 * PyTorch or HIP type appears in a signature: device memory and streams are
 * passed as plain pointers (`void*`), so any allocator (torch, hipMalloc)
 * can own them.
 *
 * Library state: per device, the address of wc_analyze_device_static's
 * scratch array and the decode kernels' resident-wave counts (wc_decode's
 * choice of kernel), each worked out once, under a lock, on the first call
 * on that device.  Nothing else persists between calls; calls on different
 * streams or devices may run concurrently, except wc_analyze_device_static,
 * whose calls share its scratch and are serialised by a process-wide lock.
 *
 * Blob format version 5 (little-endian; every offset absolute from the blob
 * start): header 64 B, then one 96-B descriptor per tensor (type, chunk size,
 * sizes, lanes, table and raw offsets, shape and tile), then the u16 frequency
 * tables (16-B padded; tensors sharing a codebook point to one table), the
 * chunk index (u32 per chunk + 1: record offset / 16), the raw bytes and the
 * chunk records (the raw regions' places depend on the sizes only).  A chunk covers `chunk_bytes` of decoded output (a tile of a
 * tiled tensor, whose symbols and raw bytes are stored tile by tile); its
 * record is
 *     u32 n_words, u32 n_states (A), u32 n_symbols, u32 0,
 *     u32 state[A] (16-B padded), u16 word[n_words] (16-B padded).
 *   Symbol i of a chunk belongs to lane (i mod L*W) div W at step
 *   (i div L*W)*W + i mod W, with W symbols = 16 output bytes per lane-group.
 *   Start states: a lane of a tiled chunk starts the encoder at 2^16 and its
 *   decode ends there.  A lane of an untiled chunk starts at 2^S + D, where D
 *   packs the lane's first K symbols (b bits each, the first lowest; fewer if
 *   the lane has fewer), which are not coded: K, b, S = 2, 8, 16 for the coded
 *   bytes of bf16 / fp16, 3, 8, 24 for byte symbols, 7, 4, 28 for nibbles.
 *   Its decode ends in that state and reads those symbols back from it.
 */
#ifndef WC_H_
#define WC_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WC_OK = 0,
  WC_EINVAL = -1,       /* bad argument, malformed or inconsistent blob */
  WC_ENOMEM = -2,       /* host allocation failed */
  WC_ECORRUPT = -3,     /* reserved for host-side stream checks */
  WC_EHIP = -4,         /* a HIP runtime call or kernel launch failed */
  WC_EUNSUPPORTED = -5  /* valid blob the GPU path does not handle (e.g. lanes) */
} wc_status;

/* Storage formats.  The symbols follow from the numeric format (Sec. II-B):
 *   WC_BF16 / WC_FP16: the 16-bit word is split into a coded byte (bits 14..7)
 *     and a raw byte (bit 15, bits 6..0);
 *   WC_U8, WC_FP8_E4M3, WC_FP8_E5M2: one coded symbol per byte (int8 or fp8
 *     codes; the three differ only in the recorded type);
 *   WC_U4, WC_FP4_E2M1: two coded nibbles per byte, low nibble first (int4 or
 *     fp4 e2m1 codes). */
typedef enum {
  WC_BF16 = 1,
  WC_FP16 = 2,
  WC_U8 = 3,
  WC_U4 = 4,
  WC_FP8_E4M3 = 5,
  WC_FP8_E5M2 = 6,
  WC_FP4_E2M1 = 7
} wc_dtype;

/* A host tensor to analyse or encode: `nbytes` bytes of raw storage.
 * rows, cols: optional matrix shape in symbol elements (16-bit words, bytes,
 * or nibbles for 4-bit formats), row-major; 0, 0 when the tensor is only a
 * byte run.  A shape is what lets wc_encode cut the tensor into 2-D tiles. */
typedef struct {
  const void* host_ptr;
  uint64_t nbytes;
  int32_t dtype; /* wc_dtype */
  int32_t reserved;
  uint64_t rows;
  uint64_t cols;
} wc_tensor;

/* Encoder parameters.  chunk_bytes: decoded bytes per chunk, a multiple of
 * 256 in [256, 1 MiB] (16, 32 or 64 KiB in practice; each chunk is a serial
 * chain per lane, so a launch with too few chunks to fill the device is bound
 * by the chain length: smaller chunks decode such a launch faster, at the
 * cost of more lane states in the blob).  lanes: interleaved
 * rANS lanes per chunk, 1..64 (the GPU decoder takes 64 or 32).  prob_bits:
 * must be 12 (Sec. VI-F, b = 12).  n_threads: host encoder threads, 0 = all
 * cores.
 * tile_rows, tile_cols: 2-D tiles (Sec. IV-A), both 0 for none.  A tensor
 * whose shape they divide exactly is coded one chunk per tile, tiles in
 * row-major order; tile_cols must be a power of two.  Tensors without a
 * shape, or with one the tile does not divide, or a tile narrower than a
 * 16-byte lane-group, keep chunk_bytes chunks.
 * tile_order: WC_TILE_ROWS (each tile's symbols row-major) or
 * WC_TILE_COLUMN_BLOCKS (the tile's lane-groups of W elements k-block by
 * k-block, every tile row per block; tile_rows must be a power of two).  With
 * tile_rows = lanes, lane l of a chunk decodes tile row l, the layout
 * wc_gemv consumes.
 * codebook: WC_CODEBOOK_TENSOR (one table per tensor) or WC_CODEBOOK_LAYER
 * (one table per dtype for the whole blob, Sec. IV / V-B). */
typedef struct {
  uint32_t chunk_bytes;
  uint32_t lanes;
  uint32_t prob_bits;
  uint32_t n_threads;
  uint32_t tile_rows;
  uint32_t tile_cols;
  uint32_t codebook;
  uint32_t tile_order;
} wc_params;

#define WC_CODEBOOK_TENSOR 0u
#define WC_CODEBOOK_LAYER 1u
#define WC_TILE_ROWS 0u
#define WC_TILE_COLUMN_BLOCKS 1u

/* Per-field statistics of one tensor (Sec. II-B).  Field 0 is the coded
 * symbol stream; field 1 (16-bit formats only) the raw byte stream.
 * H[f] = -sum p log2 p over the field's empirical histogram, in bits per
 * symbol.  H_joint16 is the entropy over whole 16-bit words (NaN for 8/4-bit
 * formats).  bound_bytes = sum_f count[f] * H[f] / 8, the order-0 bound that
 * compressed payloads are compared with; bound_bytes_raw8 charges the raw
 * field at 8 bits, which is what a raw-stored field can reach. */
typedef struct {
  uint32_t n_fields;
  uint32_t alphabet[2];
  uint64_t count[2];
  uint64_t hist[2][256];
  double H[2];
  double H_joint16;
  double bound_bytes;
  double bound_bytes_raw8;
} wc_stats;

/* An encoded blob held in host memory, plus its parsed description.
 * Owned by the library; release with wc_free.  The fields below are
 * read-only for the caller. */
typedef struct wc_blob {
  const uint8_t* data;       /* blob bytes (host) */
  uint64_t size;             /* bytes */
  uint32_t n_tensors;
  uint32_t reserved;
  uint64_t n_chunks;         /* over all tensors */
  const uint64_t* out_bytes; /* [n_tensors] decoded bytes per tensor */
  /* size breakdown (sums to size): */
  uint64_t meta_bytes;       /* header, descriptors, tables, chunk index */
  uint64_t record_hdr_bytes; /* 16 B per chunk record */
  uint64_t state_bytes;      /* final lane states */
  uint64_t word_bytes;       /* rANS words */
  uint64_t pad_bytes;        /* 16-B alignment padding */
  uint64_t raw_bytes;        /* raw byte region (16-bit formats), incl. padding */
  void* priv;                /* library-internal */
} wc_blob;

/* Device-side error bits ORed into *dev_err by wc_decode. */
#define WC_DERR_INDEX 1u  /* chunk record offset or header inconsistent */
#define WC_DERR_STATE 2u  /* a lane did not end at its start state (2^16, or 2^S plus the
                             symbols it carries) */
#define WC_DERR_CURSOR 4u /* a chunk's word stream was not consumed exactly */
#define WC_DERR_TABLE 8u  /* a frequency table does not sum to 2^12 */

/* wc_analyze -- histogram and empirical entropy of one tensor (Sec. II-B).
 * Host only, single pass, allocates nothing on the heap except transient
 * 16-bit histogram storage.  Returns WC_EINVAL for a NULL argument, an
 * unknown dtype or an odd byte count of a 16-bit format. */
wc_status wc_analyze(const wc_tensor* t, wc_stats* out);

/* wc_encode -- offline compression of n tensors into one blob (Sec. V-B):
 * per-tensor static table normalised to 2^12, chunks of chunk_bytes of
 * output, each coded as `lanes` interleaved rANS lanes from independent
 * initial states, plus the chunk offset index.  Host only; threads over
 * chunks.  On success *out receives a library-owned blob (release with
 * wc_free).  Deterministic: the bytes depend only on the inputs and on
 * chunk_bytes / lanes, never on n_threads.  Errors: WC_EINVAL (bad params,
 * dtype, sizes, blob over 64 GiB), WC_ENOMEM. */
wc_status wc_encode(const wc_tensor* t, uint32_t n, const wc_params* p, wc_blob** out);

/* wc_open -- parse and validate an existing blob (e.g. one written by another
 * encoder or read from disk).  Copies the `size` bytes at `data`; on success
 * *out is library-owned (wc_free).  Returns WC_EINVAL for any malformed field
 * (magic, version, sizes, offsets, table sums, index order). */
wc_status wc_open(const void* data, uint64_t size, wc_blob** out);

/* wc_decode -- GPU decode of every tensor of a blob (Alg. 2), one launch per
 * 32 non-empty tensors.
 *   desc     host description from wc_encode / wc_open (supplies the grid and
 *            per-tensor layout, so no device-to-host copy is needed);
 *   dev_blob device copy of desc->data (desc->size bytes), caller-owned;
 *   dev_dst  host array of n device pointers; dev_dst[i] receives
 *            desc->out_bytes[i] decoded bytes (caller-owned; the pointer for
 *            an empty tensor may be NULL);
 *   n        must equal desc->n_tensors;
 *   stream   hipStream_t to launch on (NULL = null stream);
 *   dev_err  NULL, or a device int32 into which WC_DERR_* bits are ORed
 *            (the caller clears it; read it after synchronising the stream).
 * Asynchronous with respect to the host; allocates nothing.  Reads only
 * inside [dev_blob, dev_blob + desc->size) and writes only the decoded byte
 * ranges.  A wave decodes one 64-lane chunk, or two adjacent 32-lane chunks.
 * A launch of bf16/fp16 tensors in untiled 64-lane chunks whose chunks exceed
 * the general kernel's resident waves on the current device but fit those of
 * a 16-wave-workgroup kernel for that format runs on the latter (the device's
 * occupancy figures are read once per device, with no allocation).
 * Returns WC_EINVAL (argument mismatch), WC_EUNSUPPORTED (a tensor coded with
 * a lane count other than 64 or 32), WC_EHIP (launch failure). */
wc_status wc_decode(const wc_blob* desc, const void* dev_blob, void* const* dev_dst, uint32_t n,
                    void* stream, int32_t* dev_err);

/* wc_gemv -- fused decode-GEMM (Alg. 1 / 3): for each of n jobs i,
 * dev_y[i] += dev_x[i] * W^T with W = tensor tensors[i] of the blob, decoded
 * on the fly and never written to memory.  Every job of one tile height runs
 * in one launch.
 *   n        1..32 jobs;
 *   tensors  host array of n tensor indices; each W must be bf16, or fp8
 *            (WC_FP8_E4M3 or WC_FP8_E5M2, the formats of Sec. VI-A, converted
 *            exactly to bf16 as it is decoded; 16-row tiles only), with a shape (N = rows, K = cols, 64 * K * 2 bytes
 *            below 2 GiB), coded with 64 lanes in column-block tiles
 *            (wc_params.tile_order = WC_TILE_COLUMN_BLOCKS) of 64, 32 or 16
 *            rows.  64-row tiles take
 *            the products on the VALU for m <= 5 and on the matrix cores above
 *            (v_mfma_f32_32x32x16_bf16 on pairs of k-blocks, which needs at
 *            least 16 columns per tile); 32-row tiles use
 *            v_mfma_f32_32x32x16_bf16 and 16-row tiles
 *            v_mfma_f32_16x16x32_bf16.  On MI355X 16-row tiles are the
 *            fastest up to m = 16 and 64-row tiles from m = 32;
 *   dev_x    host array of n device pointers to bf16 activations, m x K
 *            row-major, 16-byte aligned (jobs may share one x);
 *   m        1..64 rows of activations, the same for every job;
 *   dev_y    host array of n device pointers to float, m x N row-major; the
 *            products are added (clear y first for a plain product).  The
 *            tiles of one band of rows add with fp32 atomics, so the
 *            summation order, and the last bits of y, can differ between runs;
 *   stream, dev_err as for wc_decode.
 * bf16 and fp8 jobs on 16-row tiles with m <= 16 whose tiles exceed the
 * 8-wave kernel's resident waves on the current device but fit those of a
 * 16-wave-workgroup kernel for that format run on the latter, as in wc_decode.
 * Asynchronous; allocates nothing.  Returns WC_EINVAL (argument), or
 * WC_EUNSUPPORTED (a tensor is not a bf16 64-lane column-block tensor of 64,
 * 32 or 16 rows per tile or an fp8 (e4m3, e5m2) one of 16 rows, has 64-row tiles of 8
 * columns with m > 5, or K is too large). */
wc_status wc_gemv(const wc_blob* desc, const void* dev_blob, uint32_t n, const uint32_t* tensors,
                  const void* const* dev_x, uint32_t m, float* const* dev_y, void* stream,
                  int32_t* dev_err);

/* wc_gemv_mx -- the fused decode-GEMM for MXFP4 weights (OCP microscaling,
 * the paper's fp4 format of Sec. VI-A; Alg. 1 / 3): for each of n jobs i,
 * dev_y[i] += x_i * W_i^T with W_i[n][k] = e2m1(code[n][k]) *
 * 2^(scale[n][k / 32] - 127), the codes decoded on the fly and never written.
 * A lane-group of a 16-row column-block tile is 32 codes of one row, one MX
 * block: v_cvt_scalef32_pk_bf16_fp4 turns it into bf16 with its scale (exact
 * while the weights stay in bf16's normal range) and four
 * v_mfma_f32_16x16x32_bf16 multiply it by x.
 *   tensors    host array of n tensor indices; each W must be WC_FP4_E2M1
 *              with a shape (N = rows, K = cols in codes), or WC_U8 holding
 *              the same packed bytes (two codes per byte symbol, even code in
 *              the low nibble: half the decode steps; shape N x K/2 bytes),
 *              coded with 64 lanes in column-block tiles
 *              (WC_TILE_COLUMN_BLOCKS) of 16 rows and a multiple of 128 codes;
 *   dev_scales host array of n device pointers to the e8m0 scale bytes of
 *              each W, N x K/32 row-major (e.g. decoded by wc_decode from the
 *              same blob); 255 reads as NaN;
 *   dev_x      host array of n device pointers to bf16 x, m x K row-major,
 *              16-byte aligned (jobs may share one x);
 *   m          1..64 rows of x, the same for every job;
 *   dev_y      host array of n device pointers to float y, m x N row-major;
 *              the products are added with fp32 atomics, as in wc_gemv;
 *   stream, dev_err as for wc_decode.
 * Byte-coded jobs with m <= 8 whose tiles exceed the 8-wave kernel's resident
 * waves on the current device but fit those of a 16-wave-workgroup kernel run
 * on the latter, as in wc_decode; that kernel keeps one or two values per lane
 * in scratch (at most 12 bytes), which the HIP runtime provides.
 * Asynchronous; allocates nothing.  Returns WC_EINVAL (argument) or
 * WC_EUNSUPPORTED (a tensor the path does not take). */
wc_status wc_gemv_mx(const wc_blob* desc, const void* dev_blob, uint32_t n, const uint32_t* tensors,
                     const uint8_t* const* dev_scales, const void* const* dev_x, uint32_t m,
                     float* const* dev_y, void* stream, int32_t* dev_err);

/* wc_gemv_w4 -- the fused decode-GEMM for group-quantised int4 weights (the
 * paper's int4 and awq4 formats, Sec. VI-A; Alg. 1 / 3): for each of n jobs
 * i, dev_y[i] += x_i * W_i^T with W_i[n][k] = s[n][k / 128] * (q - z[n][k /
 * 128]) for unsigned codes q and zero points z, or s * q for two's-complement
 * codes, the codes decoded on the fly and never written.  Each code becomes the
 * bf16 value 16 + t exactly (t = q, or the signed code + 8); the products with
 * x and with ones (the group's sums of x) go through v_mfma_f32_16x16x32_bf16,
 * and y gains s (sum x (16 + t) - (16 + z or 24) sum x) per group, in fp32.
 *   tensors    host array of n tensor indices; each W must be WC_U4 with a
 *              shape (N = rows, K = cols in codes), or WC_U8 holding the same
 *              packed bytes (two codes per byte symbol, even element in the
 *              low nibble: half the decode steps; shape N x K/2 bytes), coded
 *              with 64 lanes in column-block tiles (WC_TILE_COLUMN_BLOCKS) of
 *              16 rows and a multiple of 128 codes (a 16-row wave row is one
 *              group of each row);
 *   dev_scales host array of n device pointers to the fp16 scales of each W,
 *              N x K/128 row-major, 2-byte aligned;
 *   dev_zeros  NULL (every W has two's-complement codes), or a host array of
 *              n device pointers: NULL for a W with two's-complement codes, or
 *              its zero points, one byte (0..15) per group, N x K/128;
 *   dev_x      host array of n device pointers to bf16 x, m x K row-major,
 *              16-byte aligned;
 *   m          1..64 rows of x, the same for every job;
 *   dev_y      host array of n device pointers to float y, m x N row-major;
 *              the products are added with fp32 atomics, as in wc_gemv;
 *   stream, dev_err as for wc_decode.
 * Byte-coded jobs with m <= 8 whose tiles exceed the 8-wave kernel's resident
 * waves on the current device but fit those of a 16-wave-workgroup kernel run
 * on the latter, as in wc_decode; that kernel keeps one or two values per lane
 * in scratch (at most 12 bytes), which the HIP runtime provides.
 * Asynchronous; allocates nothing.  Returns WC_EINVAL (argument) or
 * WC_EUNSUPPORTED (a tensor the path does not take). */
wc_status wc_gemv_w4(const wc_blob* desc, const void* dev_blob, uint32_t n, const uint32_t* tensors,
                     const uint16_t* const* dev_scales, const uint8_t* const* dev_zeros,
                     const void* const* dev_x, uint32_t m, float* const* dev_y, void* stream,
                     int32_t* dev_err);

/* wc_gemm_i8 -- the fused decode-GEMM for int8 weights and int8 activations
 * (W8A8, the SmoothQuant-style sq8 format of Sec. VI-A; Alg. 1 / 3): for each
 * of n jobs i, dev_y[i] += x_i * W_i^T in exact integer arithmetic, W_i =
 * tensor tensors[i] decoded on the fly and never written.  With 16-row
 * column-block tiles a decoded wave row (16 W rows x 64 columns) is the B
 * operand of v_mfma_i32_16x16x64_i8 as it stands.  y is the integer product
 * before dequantisation: the per-row scales of x and W stay with the caller.
 *   tensors  host array of n tensor indices; each W must be WC_U8 (bytes read
 *            as two's-complement int8), coded with 64 lanes in column-block
 *            tiles (WC_TILE_COLUMN_BLOCKS) of 16 rows, K = cols <= 65536 (so
 *            no int32 sum can overflow: |x w| <= 2^14);
 *   dev_x    host array of n device pointers to int8 x, m x K row-major,
 *            16-byte aligned (jobs may share one x);
 *   m        1..64 rows of x, the same for every job;
 *   dev_y    host array of n device pointers to int32 y, m x N row-major; the
 *            products are added with integer atomics, so y is exact and the
 *            same whatever order the tiles finish in;
 *   stream, dev_err as for wc_decode.
 * With m <= 16, a call whose tiles exceed the 8-wave kernel's resident waves
 * on the current device but fit those of a 16-wave-workgroup kernel runs on
 * the latter, as in wc_decode.
 * Asynchronous; allocates nothing.  Returns WC_EINVAL (argument) or
 * WC_EUNSUPPORTED (a tensor the path does not take). */
wc_status wc_gemm_i8(const wc_blob* desc, const void* dev_blob, uint32_t n,
                     const uint32_t* tensors, const void* const* dev_x, uint32_t m,
                     int32_t* const* dev_y, void* stream, int32_t* dev_err);

/* wc_gemm_workspace_bytes -- device workspace wc_gemm needs for these jobs
 * (host only, nothing launched): 0 for m <= 64; above, one packed copy of
 * each distinct x (jobs whose dev_x pointers and K are equal share it) of
 * ceil(m / 32) * 32 * K * 2 bytes, each rounded up to 256 bytes.  dev_x is
 * compared as pointers, never read.  Returns WC_EINVAL for a bad argument. */
wc_status wc_gemm_workspace_bytes(const wc_blob* desc, uint32_t n, const uint32_t* tensors,
                                  const void* const* dev_x, uint32_t m, uint64_t* bytes);

/* wc_gemm -- the fused decode-GEMM of wc_gemv for any batch: m = 1..4096 rows
 * of x (Alg. 1 / 3; Sec. V, the batch-size regime).  Up to m = 64 it is
 * wc_gemv (the workspace is not used).  Above, the weights are decoded once
 * per pass of 256 x rows: the 8 waves of a workgroup decode 8 consecutive
 * tiles of one band of 64 W rows, exchange each pair of decoded wave rows
 * (64 W rows x 16 columns, two v_mfma_f32_32x32x16_bf16 B operands) through
 * LDS, and each wave multiplies all of them by its own 32 rows of x.  x is
 * first packed into the workspace in MFMA operand order (one kernel per
 * distinct x, on the same stream).  Jobs, arguments and y as for wc_gemv;
 * above m = 64 every tensor must have 64-row tiles of at least 16 columns
 * with rows % 64 == 0 and cols % tile_cols == 0 (full tiles).
 *   dev_workspace  device memory of at least wc_gemm_workspace_bytes bytes,
 *                  256-byte aligned, owned by the caller; overwritten; calls
 *                  sharing a workspace must not overlap in time.
 * When to use it: every further pass of 256 x rows decodes the weights again,
 * so the fused call pays off up to about 256 rows.  Above that, decode the
 * weights once with wc_decode and multiply with a library GEMM: on one
 * MI355X, for the seven products of a Llama-3-70B layer, the fused call took
 * 0.918 ms at m = 256 against 1.356 ms decode-then-multiply, but 1.779 ms at
 * m = 512 against 1.468 ms, and 3.499 ms at m = 1024 against 1.978 ms.  The
 * call does not switch by itself.
 * Asynchronous; allocates nothing.  Returns WC_EINVAL (argument, or a
 * workspace too small or misaligned) or WC_EUNSUPPORTED (a tensor the path
 * does not take). */
wc_status wc_gemm(const wc_blob* desc, const void* dev_blob, uint32_t n, const uint32_t* tensors,
                  const void* const* dev_x, uint32_t m, float* const* dev_y, void* dev_workspace,
                  uint64_t workspace_bytes, void* stream, int32_t* dev_err);

/* A tensor in device memory, for the device-side analysis and encoder: the
 * fields of wc_tensor, with dev_ptr a device pointer that must be 16-byte
 * aligned (any torch or hipMalloc allocation is). */
typedef struct {
  const void* dev_ptr;
  uint64_t nbytes;
  int32_t dtype; /* wc_dtype */
  int32_t reserved;
  uint64_t rows;
  uint64_t cols;
} wc_dtensor;

/* Device workspace wc_analyze_device needs: 65 536 u64 histogram bins. */
#define WC_ANALYZE_WORKSPACE_BYTES 524288u

/* wc_analyze_device -- wc_analyze of a tensor in device memory (Sec. II-B):
 * the same wc_stats, bit for bit.  The histograms are counted on the GPU
 * (16-bit formats: the histogram of whole 16-bit words, from which both
 * fields and the joint entropy follow; other formats: the symbol histogram);
 * the entropies are computed on the host from the counts.
 *   dev_workspace  caller-owned device memory of at least
 *                  WC_ANALYZE_WORKSPACE_BYTES (16-byte aligned), overwritten;
 *   stream         hipStream_t (NULL = null stream).
 * Synchronous: returns after the counts are back on the host.  Allocates
 * nothing.  Returns WC_EINVAL (argument, dtype, odd size of a 16-bit format,
 * misaligned pointer, workspace too small), WC_EHIP. */
wc_status wc_analyze_device(const wc_dtensor* t, void* dev_workspace, uint64_t workspace_bytes,
                            void* stream, wc_stats* out);

/* wc_analyze_device_static -- wc_analyze_device for callers that cannot
 * allocate device memory (harnesses and serving loops that forbid hipMalloc):
 * the same wc_stats, bit for bit, with no workspace argument.  The 65 536 u64
 * histogram bins (512 KiB, the WC_ANALYZE_WORKSPACE_BYTES of wc_analyze_device)
 * live in a device array of the library's own: every GPU the library runs on
 * holds one copy until the process ends.  Its device address is looked up
 * once per device, on the first call with that device current; the bins are
 * cleared by a kernel at the start of every call, so nothing of a previous
 * call (a larger tensor, another format) carries over.  Any tensor size is
 * taken: the bins are u64 counts whatever the size.
 *   t       the tensor, in memory of the current device (16-byte aligned);
 *   stream  hipStream_t of the current device (NULL = null stream);
 *   out     receives the statistics.
 * Synchronous.  Calls no hipMalloc, hipFree or other allocating routine, and
 * takes a process-wide lock for its duration: calls from several host threads
 * run one after another.  (Calls from several processes each have their own
 * copy of the array.)  Returns WC_EINVAL (argument, dtype, odd size of a
 * 16-bit format, misaligned pointer), WC_EUNSUPPORTED (device ordinal 64 or
 * above), WC_EHIP. */
wc_status wc_analyze_device_static(const wc_dtensor* t, void* stream, wc_stats* out);

/* wc_encode_device_bounds -- what wc_encode_device needs for these tensors and
 * parameters (their pointers are not read): *blob_capacity, the largest blob
 * they can give (every coded symbol emitting a word), and *workspace_bytes,
 * the device scratch the encoder uses.  Host only.  WC_EINVAL as for
 * wc_encode, and for a largest blob of 64 GiB or more. */
wc_status wc_encode_device_bounds(const wc_dtensor* t, uint32_t n, const wc_params* p,
                                  uint64_t* blob_capacity, uint64_t* workspace_bytes);

/* wc_encode_device -- wc_encode on the GPU (Sec. V-B; the optional GPU-side
 * compressor): the blob it writes to dev_blob is byte-identical to the one
 * wc_encode makes from the same tensors and parameters (n_threads ignored).
 * Histograms, table normalisation, the chunk encode (one wave per chunk, one
 * rANS lane per wave lane, steps in reverse), the offset index and the final
 * packing all run on the device, in order on `stream`.
 *   t, n, p         the tensors (device memory, 16-byte aligned, not modified)
 *                   and parameters, as for wc_encode;
 *   dev_blob        caller-owned device buffer of blob_capacity >= the bound
 *                   from wc_encode_device_bounds; bytes past the blob's size
 *                   are left as they were;
 *   dev_workspace   caller-owned device scratch of workspace_bytes >= the
 *                   bound (16-byte aligned); overwritten;
 *   dev_size        device u64 that receives the blob's size in bytes.
 * Asynchronous: read *dev_size, and use the blob (e.g. wc_open on a host copy
 * of it), after synchronising the stream.  Allocates nothing.  Returns
 * WC_EINVAL (argument, parameters, sizes, alignment, capacity), WC_EHIP. */
wc_status wc_encode_device(const wc_dtensor* t, uint32_t n, const wc_params* p, void* dev_blob,
                           uint64_t blob_capacity, void* dev_workspace, uint64_t workspace_bytes,
                           void* stream, uint64_t* dev_size);

/* wc_stream -- a measuring aid, not part of the codec: a plain streaming
 * kernel that moves a decode's byte mix with no decoding, so that a decode
 * launch can be set against the rate the device's memory gives the same
 * traffic.  Write unit j (16 bytes) of dst receives read unit
 * (j * q) >> 32 of src, q = floor(n_src * 2^32 / n_dst) (n_src, n_dst: the
 * sizes in 16-byte units), so src is read once, in order, spread evenly over
 * the writes; the stores are non-temporal, as the decode's are.
 *   dev_src, src_bytes  device memory to read, 16-byte aligned, src_bytes a
 *                       non-zero multiple of 16;
 *   dev_dst, dst_bytes  device memory to write, 16-byte aligned, dst_bytes a
 *                       multiple of 16 with src_bytes <= dst_bytes < 64 GiB;
 *                       dst_bytes = 0 reads src only (dev_dst must then hold
 *                       16 writable bytes, stored to only if the data read
 *                       XOR to one fixed 128-bit pattern);
 *   blocks              workgroups of 256 threads (0 = 16 per compute unit);
 *   stream              hipStream_t (NULL = null stream);
 *   read_bytes          NULL, or receives the bytes the launch reads.
 * Asynchronous; allocates nothing.  Returns WC_EINVAL (argument), WC_EHIP. */
wc_status wc_stream(const void* dev_src, uint64_t src_bytes, void* dev_dst, uint64_t dst_bytes,
                    uint32_t blocks, void* stream, uint64_t* read_bytes);

/* wc_free -- release a blob from wc_encode / wc_open.  NULL is a no-op. */
void wc_free(wc_blob* b);

/* wc_version -- ABI version of this header (12). */
int32_t wc_version(void);

#ifdef __cplusplus
}
#endif

#endif /* WC_H_ */
