/*
 * sllm.h — C ABI of the MI355X checkpoint loader.
 *
 * The library converts a tensor checkpoint into a loading-optimized format
 * and streams it from pinned host DRAM into one preallocated HBM buffer
 * (ServerlessLLM, Sec. 4, fast multi-tier checkpoint loading).
 *
 * Format (Sec. 4.1).  A checkpoint directory holds two files:
 *   sllm.part0  the partition for one GPU: the tensors' bytes only, in the
 *               caller's order, each at an offset aligned to A (a power of
 *               two), zero padding between tensors, zero-filled up to
 *               F = align_up(T, 4096) bytes, where T = sum align_up(s_i, A).
 *   sllm.index  the tensor index: name -> (dtype, shape, partition, offset,
 *               size), little-endian, closed by a CRC-32 (IEEE).  The exact
 *               byte layout is in docs/FORMAT.md.
 * A tensor's device address is base + offset (Sec. 4.1, direct tensor
 * addressing).
 *
 * Loading (Sec. 4.2).  Chunk k of a partition is the byte range
 * [kC, min(kC + C, T)).  Chunks move through a pool of fixed-size pinned host
 * chunks (the DRAM tier, with allocate/evict calls under application control)
 * and from there into device memory, either by the copy (SDMA) engines or by
 * a gfx950 kernel that reads the mapped host chunks directly.
 *
 * Conventions.
 *   - Every call returns an int32_t status: SLLM_OK (0) or a negative
 *     SLLM_E_* code; sllm_last_error() then gives a message for this thread.
 *   - No C++ exception crosses this interface.
 *   - "Device pointer" means an address in the HIP device's memory (for
 *     example a torch uint8 CUDA tensor's data_ptr()); "stream" is a
 *     hipStream_t passed as void* (NULL = the null stream).
 *   - The caller owns every buffer and stream it passes in.  The library
 *     owns its handles and everything reachable from them until the matching
 *     close/destroy call.
 *   - A handle may be used by one thread at a time; different handles may
 *     be used from different threads.
 *   - Copy streams (and their fork/join events) outlive the handles that
 *     used them: a closed handle leaves its idle streams to the next handle
 *     on the same device (at most 32 sets per process, kept until the
 *     process ends), so opening a handle per load costs no stream creation.
 *     A caller that resets a device must not use the library afterwards.
 *   - Reader threads outlive the loads that start them: a finished reader
 *     waits idle (at most 64 per process, until the process ends) for the
 *     next load or pool fill, which then wakes it instead of starting a
 *     thread.
 *
 * Environment (read by the library; none is needed for normal use).
 *   SLLM_LOG_LEVEL        0 quiet (default), 1 info, 2 debug, on stderr.
 *   SLLM_TRACE_FILE       streamed loads append each chunk's read, move and
 *                         done times to this CSV file.
 *   SLLM_ROCTX=1          host stages become roctx ranges (rocprofv3
 *                         --marker-trace); the roctx library is loaded then.
 *   SLLM_READ_STREAM=0    buffered chunks are read straight into pinned
 *                         memory (default: through a 1 MiB per-thread buffer
 *                         copied on with streaming stores, so that the GPU
 *                         reads them from DRAM, not from dirty CPU caches).
 *   SLLM_READ_MAPPED=1    buffered files are mapped and chunks copied with
 *                         streaming stores instead of read with pread.
 *   SLLM_BATCH_TARGET_MB  bytes a streamed gather batch collects (64).
 *   SLLM_SPLIT_CHUNKS     leading chunks of a streamed load that all readers
 *                         read together in pieces (one per I/O thread; 0
 *                         reads every chunk whole).
 *   SLLM_IDLE_WORKERS     idle reader threads kept for later loads (64; 0
 *                         starts every reader on a new thread).
 *   SLLM_SDMA_MAX_COPY_MB largest merged copy-engine copy of cached chunks (256).
 *   SLLM_POOL_ARENA_MB    size of each pinned allocation a pool is cut from (1024).
 *   SLLM_K1_BLOCKS, SLLM_K1_STREAM_BLOCKS, SLLM_K1_UNROLL, SLLM_K1_NT,
 *   SLLM_K2_NT, SLLM_K2_MAX_GRID, SLLM_K2_UNROLL, SLLM_NOALLOC_PLAN_BLOCKS
 *                         kernel launch shapes, read at every launch (for
 *                         measurements and tests; the defaults are tuned).
 */
#ifndef SLLM_H
#define SLLM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes -------------------------------------------------------- */
#define SLLM_OK          0
#define SLLM_E_INVAL    -1  /* bad argument or option                           */
#define SLLM_E_IO       -2  /* a file could not be opened, read or written      */
#define SLLM_E_FORMAT   -3  /* index or partition damaged or inconsistent       */
#define SLLM_E_NOMEM    -4  /* host or pool memory exhausted                    */
#define SLLM_E_HIP      -5  /* a HIP runtime call failed                        */
#define SLLM_E_RANGE    -6  /* destination buffer too small                     */
#define SLLM_E_BUSY     -7  /* object in use (load in progress, cached, opened) */
#define SLLM_E_NOTFOUND -8  /* no such tensor / checkpoint                      */

/* ---- dtypes (stored bytes are never converted) ---------------------------- */
#define SLLM_DTYPE_F32  0
#define SLLM_DTYPE_F16  1
#define SLLM_DTYPE_BF16 2
#define SLLM_DTYPE_I8   3
#define SLLM_MAX_NDIM   8

/* =========================================================================
 * Conversion (Sec. 4.1: checkpoints are converted once, loaded many times)
 * ========================================================================= */

/* One tensor of the source checkpoint.  `data` holds `nbytes` raw
 * little-endian bytes, and nbytes must equal prod(shape) * itemsize(dtype)
 * (a 0-d tensor has one element).  `name` is non-empty UTF-8 of at most
 * 65535 bytes, unique within the checkpoint. */
typedef struct sllm_src_tensor {
    const char*    name;
    uint32_t       dtype;   /* SLLM_DTYPE_* */
    uint32_t       ndim;    /* 0 .. SLLM_MAX_NDIM */
    const int64_t* shape;   /* ndim entries, each >= 0 (may be NULL if ndim == 0) */
    const void*    data;    /* host memory; may be NULL if nbytes == 0 */
    uint64_t       nbytes;
} sllm_src_tensor;

#define SLLM_CONVERT_FSYNC 1u   /* fsync both files before returning */

typedef struct sllm_convert_opts {
    uint64_t alignment;   /* A: power of two >= 1; 0 means 256            */
    uint64_t chunk_size;  /* default load chunk size C >= 1; 0 means 16 MiB */
    uint32_t flags;       /* SLLM_CONVERT_*                                */
    uint32_t reserved;    /* must be 0                                     */
} sllm_convert_opts;

/* Write out_dir/sllm.part0 and out_dir/sllm.index for the n tensors, in the
 * given order (out_dir must exist).  opts may be NULL (A = 256, C = 16 MiB).
 * The caller's tensor memory is only read during the call.  Existing files
 * are replaced; on error both files are removed.
 * Errors: INVAL (bad tensor or option; duplicate or empty name), IO. */
int32_t sllm_convert(const sllm_src_tensor* tensors, uint64_t n,
                     const char* out_dir, const sllm_convert_opts* opts);

/* Streaming form of sllm_convert for checkpoints that do not fit in host
 * memory twice: tensors are added one at a time and written immediately.
 * The files it produces are byte-identical to sllm_convert's.
 * sllm_writer_close writes the index and frees the writer (even on error);
 * sllm_writer_abort removes the partial files and frees the writer.
 * Errors: as sllm_convert; after a failed sllm_writer_add the writer only
 * accepts sllm_writer_abort or sllm_writer_close (which then removes the
 * files and returns the error). */
typedef struct sllm_writer sllm_writer;
int32_t sllm_writer_open(const char* out_dir, const sllm_convert_opts* opts,
                         sllm_writer** out);
int32_t sllm_writer_add(sllm_writer* w, const sllm_src_tensor* tensor);
int32_t sllm_writer_close(sllm_writer* w);
void    sllm_writer_abort(sllm_writer* w);

/* Convert safetensors shards (the format Hugging Face checkpoints ship in)
 * straight into out_dir: every tensor of every shard, in shard order and,
 * within a shard, in the order its bytes sit in the file, so each shard is
 * read front to back once.  Supported dtypes: F32, F16, BF16, I8.
 * Errors: INVAL (another dtype, more than 8 dimensions, a name repeated
 * across shards), IO, FORMAT (malformed header, data outside the file,
 * overlapping tensors, size != numel * itemsize).  On error no files remain. */
int32_t sllm_convert_safetensors(const char* const* paths, uint64_t n_paths, const char* out_dir,
                                 const sllm_convert_opts* opts);

/* =========================================================================
 * Pinned host chunk pool: the DRAM tier (Sec. 4.2, chunk-based data
 * management: fixed-size chunks, allocation and eviction under the
 * application's control)
 * ========================================================================= */

typedef struct sllm_pool sllm_pool;

/* Allocate n_chunks pinned, device-mapped host chunks of chunk_size bytes
 * (>= 1) for HIP device `device`.  Every chunk starts on a 4 KiB boundary
 * (chunks sit align_up(chunk_size, 4096) bytes apart), so direct file reads
 * can land in them.  Allocation is slow (pages are pinned); do it once,
 * outside the load path.
 * Errors: INVAL, HIP (pinned allocation failed). */
int32_t sllm_pool_create(uint64_t chunk_size, uint64_t n_chunks, int32_t device,
                         sllm_pool** out);

/* Free the pool.  BUSY while an open checkpoint handle still uses it. */
int32_t sllm_pool_destroy(sllm_pool* pool);

typedef struct sllm_pool_info {
    uint64_t chunk_size;
    uint64_t n_chunks;
    uint64_t free_chunks;
    uint64_t cached_checkpoints;
} sllm_pool_info;
/* Sizes and occupancy of the pool.  Errors: INVAL (NULL argument). */
int32_t sllm_pool_query(const sllm_pool* pool, sllm_pool_info* out);

/* Read the whole partition of checkpoint directory `dir` into pool chunks,
 * where it stays (cached in DRAM) until sllm_pool_evict.  Loads of handles
 * opened on this pool then copy from these chunks with no file I/O.
 * io_threads = 0 means 4.  flags: SLLM_OPEN_DIRECT_IO.
 * Errors: INVAL, IO, FORMAT, NOMEM (not enough free chunks), BUSY (already
 * cached).  The checkpoint is identified by the data file's device, inode,
 * size and modification time. */
int32_t sllm_pool_cache(sllm_pool* pool, const char* dir, uint32_t io_threads,
                        uint32_t flags);

/* Return a cached checkpoint's chunks to the pool.  NOTFOUND if not cached,
 * BUSY while an open handle loads from it. */
int32_t sllm_pool_evict(sllm_pool* pool, const char* dir);

/* =========================================================================
 * Open / load / index (Sec. 4.1 direct tensor addressing; Sec. 4.2 loading)
 * ========================================================================= */

#define SLLM_ENGINE_KERNEL 0u   /* gfx950 kernel reads mapped host chunks      */
#define SLLM_ENGINE_SDMA   1u   /* hipMemcpyAsync on the copy engines          */

#define SLLM_OPEN_DIRECT_IO 1u  /* O_DIRECT file reads (buffered if the file
                                   system refuses them; see stats.direct_io) */
#define SLLM_OPEN_TIMING    2u  /* time device work with HIP events (stats)   */
#define SLLM_OPEN_INDEX_ONLY 4u /* read and validate the index only: no data
                                   file, pool or device work; for processes
                                   that view a buffer another process loaded
                                   (sllm_load then returns SLLM_E_INVAL)      */
#define SLLM_OPEN_CACHE     8u  /* keep what the first load reads: it streams
                                   the file (storage -> pinned -> HBM,
                                   pipelined) into ceil(T/C) chunks of
                                   opts->pool, one per chunk, and once it has
                                   succeeded those chunks become the pool's
                                   cached copy of the checkpoint (the DRAM
                                   tier, Sec. 4.2), as after sllm_pool_cache.
                                   Needs a pool whose chunk size is C; NOMEM
                                   if it lacks free chunks.  No effect when
                                   the checkpoint is cached already.        */

typedef struct sllm_open_opts {
    uint64_t   chunk_size;     /* C for reads from the file; 0 = pool's chunk
                                  size if a pool is given, else the index's */
    uint64_t   dev_alignment;  /* 0: device layout = file layout.  Else A2, a
                                  power of two >= 16: tensor i goes to
                                  d_i = sum_{j<i} align_up(s_j, A2), zero
                                  padded, T2 = sum align_up(s_i, A2) bytes */
    sllm_pool* pool;           /* NULL: a private pool of ring_slots chunks
                                  is allocated by sllm_open                 */
    uint32_t   io_threads;     /* file-reading threads; 0 = 4               */
    uint32_t   n_streams;      /* copy streams for the SDMA engine; 0 = 2   */
    uint32_t   ring_slots;     /* chunks in flight when streaming from the
                                  file; 0 = 2 * io_threads                  */
    uint32_t   engine;         /* SLLM_ENGINE_*                             */
    uint32_t   flags;          /* SLLM_OPEN_*                               */
    int32_t    device;         /* HIP device ordinal                        */
} sllm_open_opts;

typedef struct sllm_ckpt sllm_ckpt;

/* Read and validate dir/sllm.index (magic, version, CRC, unique names,
 * sizes = numel * itemsize, aligned ordered non-overlapping offsets,
 * T = padded sum, file length F) and open dir/sllm.part0.  If `opts->pool`
 * caches this checkpoint, later loads copy from the cached chunks; else they
 * stream the file through ring_slots pool chunks.  opts may be NULL
 * (defaults above, device 0).  With a dev_alignment the handle keeps device
 * tables of 24 bytes per tensor plus 8 bytes per 16 KiB of the device image
 * (the repack kernel's plan), built here.
 * Errors: INVAL (also: direct reads where the chunk size or the padded file
 * length F is not a multiple of the file's direct-I/O alignment), IO,
 * FORMAT, NOMEM, HIP. */
int32_t sllm_open(const char* dir, const sllm_open_opts* opts, sllm_ckpt** out);

/* Bytes a load writes: T (file layout) or T2 (dev_alignment != 0); 0 for a
 * NULL handle. */
uint64_t sllm_total_bytes(const sllm_ckpt* h);

/* Load the checkpoint into device memory [dev_dst, dev_dst + total_bytes).
 * dev_dst must be 16-byte aligned.  All of [0, total) is written, padding
 * included (as zero); bytes past it are untouched.  Returns once every file
 * read has finished and every copy or kernel has been enqueued; completion is
 * ordered on `stream`: work queued there after this call sees every byte.
 * Errors: INVAL (dev_dst is not device memory of the handle's device, is
 * memory whose allocation range the runtime cannot report, or is not
 * 16-byte aligned), RANGE (dst_bytes < total, or the range runs past the
 * end of dev_dst's allocation), IO, HIP, BUSY (another load on this
 * handle).  On error, in-flight work is drained and the destination's
 * contents are unspecified; the handle stays usable. */
int32_t sllm_load(sllm_ckpt* h, void* dev_dst, uint64_t dst_bytes, void* stream);

/* On-device repack of a file-layout image into the device layout: src holds
 * the partition's first T bytes (as sllm_load writes them with
 * dev_alignment = 0) and dst receives T2 bytes laid out with the handle's
 * dev_alignment.  src and dst are device pointers, 16-byte aligned, and must
 * not overlap.  Enqueued on `stream`.
 * Errors: INVAL (handle opened without dev_alignment, overlap, a buffer that
 * is not device memory of the handle's device or whose allocation range the
 * runtime cannot report), RANGE, HIP. */
int32_t sllm_repack(const sllm_ckpt* h, const void* src_dev, uint64_t src_bytes,
                    void* dst_dev, uint64_t dst_bytes, void* stream);

/* sllm_repack for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same result, byte for byte, with no hipMalloc, hipFree or other
 * allocation.  Its device tables (sizes, file and device offsets, and the
 * repack plan for one window of the destination at a time) live in a fixed
 * library area of SLLM_NOALLOC_SCRATCH_BYTES per device, which each device
 * holds from the library's first kernel launch on it until the process
 * ends.  The sizes travel as kernel arguments; every table is rewritten by
 * each call, so nothing carries over between calls.
 *   h              any open handle, INDEX_ONLY included (its index gives the
 *                  layout); it may have been opened without a dev_alignment
 *   dev_alignment  A2, a power of two >= 16; 0 means the handle's own
 *   src_dev        the file-layout image, T = sllm_total_bytes of an
 *                  unaligned handle; src_bytes >= T
 *   dst_dev        receives T2 = sum align_up(s_i, A2) bytes; dst_bytes >= T2
 * Buffers are device memory of the handle's device, 16-byte aligned, and do
 * not overlap.  Enqueued on `stream`; the call returns without waiting.
 * Calls that overlap on one device (different streams or threads, or one
 * stream while another call's kernels still run elsewhere) race for the
 * area: order them, for example on one stream.
 * Errors: INVAL (no or bad alignment, overlap, a buffer that is not device
 * memory of the handle's device), RANGE (a buffer too small, or more than
 * SLLM_NOALLOC_MAX_TENSORS tensors), HIP. */
#define SLLM_NOALLOC_SCRATCH_BYTES (16ull << 20)
#define SLLM_NOALLOC_MAX_TENSORS   65536ull
int32_t sllm_repack_noalloc(const sllm_ckpt* h, uint64_t dev_alignment, const void* src_dev,
                            uint64_t src_bytes, void* dst_dev, uint64_t dst_bytes, void* stream);

/* One tensor of the index.  `offset` is relative to the device buffer:
 * the file offset o_i, or d_i when the handle has a dev_alignment.  `name`
 * stays valid until sllm_close. */
typedef struct sllm_tensor_info {
    const char* name;
    uint32_t    dtype;
    uint32_t    ndim;
    int64_t     shape[SLLM_MAX_NDIM];
    uint64_t    offset;
    uint64_t    nbytes;
} sllm_tensor_info;

/* Copy up to `cap` entries, in layout order, into out[] and set *n_total to
 * the number of tensors (cap = 0 with out = NULL asks for the count only).
 * Errors: INVAL (NULL handle, or out NULL with cap > 0). */
int32_t sllm_tensor_index(const sllm_ckpt* h, sllm_tensor_info* out, uint64_t cap,
                          uint64_t* n_total);

/* Look one tensor up by name.  Errors: INVAL (NULL argument), NOTFOUND. */
int32_t sllm_tensor_find(const sllm_ckpt* h, const char* name, sllm_tensor_info* out);

typedef struct sllm_stats {
    uint64_t bytes_loaded;      /* bytes written to the device by the last load  */
    uint64_t bytes_read;        /* bytes read from the file by the last load     */
    uint64_t n_chunks;          /* chunks moved by the last load                 */
    uint64_t n_launches;        /* kernel launches or copy calls of the last load */
    uint32_t engine;            /* engine used                                   */
    uint32_t direct_io;         /* 1 if the file is read with O_DIRECT           */
    uint32_t from_cache;        /* 1 if the last load came from cached chunks    */
    uint32_t io_threads;
    double   open_s;            /* wall time of sllm_open                        */
    double   load_s;            /* wall time of the last sllm_load call          */
    double   read_wait_s;       /* time the issue loop waited for file reads     */
    double   device_ms;         /* device time of the last load (TIMING flag), else -1 */
    uint64_t bytes_bounced;     /* direct-read bytes staged through a bounce buffer
                                   because the kernel refused direct transfers
                                   into the pinned chunks                      */
    double   reader_busy_s;     /* streamed loads: I/O-thread time spent reading
                                   (summed over threads)                       */
    double   reader_starved_s;  /* streamed loads: I/O-thread time spent waiting
                                   for a free slot (summed over threads)       */
} sllm_stats;
/* Counters of the handle's last load.  With SLLM_OPEN_TIMING this waits for
 * that load's device work to finish (to read its events).  Errors: INVAL, HIP. */
int32_t sllm_get_stats(const sllm_ckpt* h, sllm_stats* out);

/* =========================================================================
 * Handoff to another process (Sec. 4.1: the model manager loads, the
 * inference process receives the GPU base address as an IPC handle, computes
 * base + offset from the index and synchronizes with the manager)
 * ========================================================================= */

typedef struct sllm_ipc_desc {
    uint8_t  mem_handle[64];    /* IPC handle of the allocation holding the buffer */
    uint8_t  event_handle[64];  /* IPC handle of an event recorded after the load  */
    uint64_t offset;            /* start of the buffer inside that allocation      */
    uint64_t bytes;             /* length of the buffer                            */
    int32_t  device;
    uint32_t flags;             /* SLLM_IPC_*                                      */
} sllm_ipc_desc;

/* event_handle is valid: the importer's stream waits for it on the device.
 * Without it the exporter finished the load before filling the descriptor
 * (the runtime offers no interprocess events), and the importer waits for
 * nothing. */
#define SLLM_IPC_HAS_EVENT 1u

/* Largest allocation this library shares across processes: opening handles
 * of larger allocations does not complete on the MI355X systems it was
 * tested on, so export refuses them. */
#define SLLM_IPC_MAX_ALLOCATION ((2ull << 30) - 1)

typedef struct sllm_export sllm_export;
typedef struct sllm_import sllm_import;

/* Share [dev_ptr, dev_ptr + bytes) (inside one device allocation of at most
 * SLLM_IPC_MAX_ALLOCATION bytes) with other processes: fills *desc (plain
 * bytes, safe to send through a pipe or file) and records the handoff event
 * on `stream`, after the work already queued there (typically sllm_load).
 * Where the runtime has no interprocess events, it instead waits for that
 * work to finish and leaves SLLM_IPC_HAS_EVENT clear.
 * Keep the export alive while importers use the buffer.
 * Errors: INVAL (not device memory, allocation too large, range outside it), HIP. */
int32_t sllm_export_create(const void* dev_ptr, uint64_t bytes, int32_t device, void* stream,
                           sllm_ipc_desc* desc, sllm_export** out);
/* Release the export (its handoff event); importers must have closed their
 * mappings.  NULL is a no-op.  Always returns SLLM_OK. */
int32_t sllm_export_destroy(sllm_export* ex);

/* Map an exported buffer into this process: *dev_ptr is its start here, and
 * `stream` waits (on the device) for the exporter's handoff event, so work
 * queued on it afterwards sees the loaded bytes.  Errors: INVAL (unknown
 * flags, or offset + bytes past the end of the mapped allocation: nothing
 * stays mapped), HIP. */
int32_t sllm_import_open(const sllm_ipc_desc* desc, void* stream, void** dev_ptr, sllm_import** out);
/* Unmap; work that reads the buffer must have finished.  NULL is a no-op.
 * Errors: HIP (the mapping could not be closed; the import is freed anyway). */
int32_t sllm_import_close(sllm_import* im);

/* =========================================================================
 * Loading-time estimate (Sec. 6, estimating model loading time): a load of
 * n bytes queued behind other loads on this server finishes after q + n / b,
 * where q sums the estimates of the loads already queued (loads run one at a
 * time per server) and b is the bandwidth of the slowest tier the load
 * crosses (the tiers are pipelined).  Measured load times refine b.
 * Host-only; no device work.
 * ========================================================================= */

#define SLLM_TIER_DRAM    1u  /* pinned host DRAM -> HBM        */
#define SLLM_TIER_STORAGE 2u  /* local file -> pinned host DRAM */

typedef struct sllm_estimator sllm_estimator;

/* Initial bandwidths in bytes per second (> 0) and the weight in (0, 1] of a
 * new measurement in the running estimate (1 = keep only the latest).
 * Errors: INVAL, NOMEM. */
int32_t sllm_estimator_create(double dram_bytes_per_s, double storage_bytes_per_s, double weight,
                              sllm_estimator** out);
void    sllm_estimator_destroy(sllm_estimator* e);

/* q + n / b for a load of `bytes` crossing `tiers` (SLLM_TIER_* bits),
 * queued behind every load enqueued and not yet completed.  Errors: INVAL
 * (NULL argument, no or unknown tier bits). */
int32_t sllm_estimator_query(const sllm_estimator* e, uint64_t bytes, uint32_t tiers, double* eta_s);

/* Queue such a load: *eta_s is its estimate (as for query) and *task its id;
 * its own n / b joins q for the loads queued after it. */
int32_t sllm_estimator_enqueue(sllm_estimator* e, uint64_t bytes, uint32_t tiers, uint64_t* task,
                               double* eta_s);

/* The task's load took `seconds`: bytes / seconds updates the bandwidth of
 * its slowest tier and the task leaves the queue.  NOTFOUND for an unknown
 * task, INVAL for seconds <= 0. */
int32_t sllm_estimator_complete(sllm_estimator* e, uint64_t task, double seconds);

/* sllm_estimator_complete with the time the handle's last load took, from
 * its own counters (sllm_get_stats): open_s plus load_s, or plus the device
 * time of the load when the handle was opened with SLLM_OPEN_TIMING and that
 * is longer (a load from cached chunks returns once its work is enqueued,
 * so only the device time covers it).  With timing on, this waits for the
 * load's device work.  Errors: INVAL (NULL argument, nothing loaded yet),
 * NOTFOUND, HIP. */
int32_t sllm_estimator_complete_load(sllm_estimator* e, uint64_t task, const sllm_ckpt* h);

/* Current bandwidth estimate of one tier (bytes per second).  Errors: INVAL. */
int32_t sllm_estimator_bandwidth(const sllm_estimator* e, uint32_t tier, double* bytes_per_s);

/* Close the handle; waits for its in-flight device work first (the copy
 * streams' and, on the caller's streams, that of every load and repack the
 * handle enqueued), so that the pool chunks and device tables that work
 * reads may be reused as soon as it returns.  NULL is a no-op.
 * Errors: BUSY (a load is running on the handle). */
int32_t sllm_close(sllm_ckpt* h);

/* Message of the last failed call on this thread ("" if none). */
const char* sllm_last_error(void);
/* Static name of a status code. */
const char* sllm_strerror(int32_t code);

#ifdef __cplusplus
}
#endif
#endif /* SLLM_H */
