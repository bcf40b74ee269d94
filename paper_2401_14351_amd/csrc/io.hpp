// File access for the storage tier (Sec. 4.2, "predictable data path"):
// direct (O_DIRECT) reads into user buffers, with a labelled buffered
// fallback where the file system refuses them.  Host-only (no HIP).
#pragma once

#include <atomic>
#include <cstdint>
#include <memory>
#include <string>

namespace sllm {

struct DataFile {
    int fd = -1;
    bool direct = false;     // opened with O_DIRECT
    uint64_t dio_align = 0;  // offset/length/buffer alignment O_DIRECT needs
    uint64_t size = 0;
    uint64_t dev = 0, ino = 0, mtime_ns = 0;
    // whether direct reads may land in pinned chunks: -1 not yet known, 0 no
    // (the kernel cannot pin those pages for the transfer), 1 yes
    std::shared_ptr<std::atomic<int>> direct_into_pinned = std::make_shared<std::atomic<int>>(-1);
    // buffered files only: a read-only shared mapping of the whole file, from
    // which chunks are copied with streaming stores (see read_chunk)
    std::shared_ptr<const uint8_t> map;
};

// Open `path` read-only; with want_direct, try O_DIRECT first and fall back
// to buffered reads if the file system rejects it.
int32_t open_data(const std::string& path, bool want_direct, DataFile* out);
void close_data(DataFile* f);

// Read exactly n bytes at `off` (retrying short reads and EINTR).  Bytes
// past the end of the file are an error.
int32_t pread_full(const DataFile& f, void* buf, uint64_t n, uint64_t off, const std::string& path);

// Read one chunk into a pinned pool chunk.  With O_DIRECT the bytes go
// straight into `dst`; where the kernel refuses direct transfers into that
// memory (EFAULT: the pages cannot be pinned for I/O), they go through a
// 16 MiB aligned per-thread bounce buffer instead, and *bounced counts them.
// A buffered read goes through a 1 MiB per-thread buffer copied on with
// streaming stores (see stream_reads).  A buffered file with a mapping has
// the chunk's pages populated first (which reports a range past the end of
// the file as an I/O error instead of faulting) and then copied with
// non-temporal stores, so the destination lines are written without first
// being read.
int32_t read_chunk(const DataFile& f, void* dst, uint64_t n, uint64_t off, const std::string& path,
                   uint64_t* bounced);

// Drop the file's pages from the page cache (for cold-read measurements).
void drop_cache(const DataFile& f);

// Whether buffered files are mapped and copied with streaming stores
// (SLLM_READ_MAPPED=1) instead of read with pread.
bool mapped_reads();

// Whether buffered reads go through a small per-thread buffer and are
// copied into the destination with streaming stores (the default;
// SLLM_READ_STREAM=0 reads into the destination directly).
bool stream_reads();

}  // namespace sllm
