// Conversion to the loading-optimized format (Sec. 4.1): the tensors' bytes
// are written in the caller's order at A-aligned offsets with zero padding,
// the partition is zero-filled to whole 4 KiB blocks, and the index is
// written last.  sllm_convert is the streaming writer applied to an array,
// so both produce the same bytes.
#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cstdlib>
#include <cstring>
#include <string>
#include <unordered_set>
#include <vector>

#include "format.hpp"

using namespace sllm;

struct sllm_writer {
    std::string data_path, index_path;
    int fd = -1;
    uint64_t alignment = 256, chunk_size = 16ull << 20;
    uint32_t flags = 0;
    uint64_t cursor = 0;   // bytes of the partition written so far (buffered included)
    IndexData ix;                          // records and names so far
    std::unordered_set<std::string> names;  // for the duplicate check
    uint8_t* buf = nullptr;   // staging buffer for small writes
    size_t fill = 0;
    int32_t error = SLLM_OK;  // sticky: first failure
};

namespace {

constexpr size_t kBufBytes = 8u << 20;

int32_t write_all(int fd, const void* p, size_t n, const std::string& path) {
    const uint8_t* q = static_cast<const uint8_t*>(p);
    while (n) {
        ssize_t w = ::write(fd, q, n);
        if (w < 0) {
            if (errno == EINTR) continue;
            return fail(SLLM_E_IO, "write %s: %s", path.c_str(), std::strerror(errno));
        }
        q += w;
        n -= (size_t)w;
    }
    return SLLM_OK;
}

int32_t flush(sllm_writer* w) {
    if (!w->fill) return SLLM_OK;
    int32_t st = write_all(w->fd, w->buf, w->fill, w->data_path);
    w->fill = 0;
    return st;
}

int32_t append(sllm_writer* w, const void* p, uint64_t n) {
    const uint8_t* q = static_cast<const uint8_t*>(p);
    while (n) {
        if (w->fill == 0 && n >= kBufBytes) {  // large payloads bypass the buffer
            SLLM_TRY(write_all(w->fd, q, n, w->data_path));
            w->cursor += n;
            return SLLM_OK;
        }
        size_t k = (size_t)std::min<uint64_t>(n, kBufBytes - w->fill);
        std::memcpy(w->buf + w->fill, q, k);
        w->fill += k;
        w->cursor += k;
        q += k;
        n -= k;
        if (w->fill == kBufBytes) SLLM_TRY(flush(w));
    }
    return SLLM_OK;
}

int32_t append_zeros(sllm_writer* w, uint64_t n) {
    while (n) {
        size_t k = (size_t)std::min<uint64_t>(n, kBufBytes - w->fill);
        std::memset(w->buf + w->fill, 0, k);
        w->fill += k;
        w->cursor += k;
        n -= k;
        if (w->fill == kBufBytes) SLLM_TRY(flush(w));
    }
    return SLLM_OK;
}

void destroy(sllm_writer* w, bool remove_files) {
    if (w->fd >= 0) ::close(w->fd);
    if (remove_files) {
        ::unlink(w->data_path.c_str());
        ::unlink(w->index_path.c_str());
    }
    std::free(w->buf);
    delete w;
}

int32_t write_file(const std::string& path, const std::string& bytes, bool do_fsync) {
    std::string tmp = path + ".tmp";
    int fd = ::open(tmp.c_str(), O_WRONLY | O_CREAT | O_TRUNC | O_CLOEXEC, 0644);
    if (fd < 0) return fail(SLLM_E_IO, "open %s: %s", tmp.c_str(), std::strerror(errno));
    int32_t st = write_all(fd, bytes.data(), bytes.size(), tmp);
    if (st == SLLM_OK && do_fsync && ::fsync(fd) != 0) st = fail(SLLM_E_IO, "fsync %s: %s", tmp.c_str(), std::strerror(errno));
    ::close(fd);
    if (st == SLLM_OK && ::rename(tmp.c_str(), path.c_str()) != 0)
        st = fail(SLLM_E_IO, "rename %s: %s", tmp.c_str(), std::strerror(errno));
    if (st != SLLM_OK) ::unlink(tmp.c_str());
    return st;
}

}  // namespace

extern "C" int32_t sllm_writer_open(const char* out_dir, const sllm_convert_opts* opts, sllm_writer** out) try {
    clear_error();
    if (!out_dir || !out) return fail(SLLM_E_INVAL, "out_dir and out must be non-NULL");
    *out = nullptr;
    auto* w = new (std::nothrow) sllm_writer;
    if (!w) return fail(SLLM_E_NOMEM, "out of host memory");
    if (opts) {
        if (opts->reserved != 0 || (opts->flags & ~SLLM_CONVERT_FSYNC)) {
            delete w;
            return fail(SLLM_E_INVAL, "unknown convert flags");
        }
        if (opts->alignment) w->alignment = opts->alignment;
        if (opts->chunk_size) w->chunk_size = opts->chunk_size;
        w->flags = opts->flags;
    }
    if (!is_pow2(w->alignment)) {
        delete w;
        return fail(SLLM_E_INVAL, "alignment %llu is not a power of two", (unsigned long long)w->alignment);
    }
    w->data_path = std::string(out_dir) + "/" + kDataName;
    w->index_path = std::string(out_dir) + "/" + kIndexName;
    if (posix_memalign(reinterpret_cast<void**>(&w->buf), 4096, kBufBytes) != 0) {
        delete w;
        return fail(SLLM_E_NOMEM, "out of host memory");
    }
    ::unlink(w->index_path.c_str());  // a stale index must not describe the new partition
    w->fd = ::open(w->data_path.c_str(), O_WRONLY | O_CREAT | O_TRUNC | O_CLOEXEC, 0644);
    if (w->fd < 0) {
        int32_t st = fail(SLLM_E_IO, "open %s: %s", w->data_path.c_str(), std::strerror(errno));
        destroy(w, false);
        return st;
    }
    *out = w;
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_writer_add(sllm_writer* w, const sllm_src_tensor* t) try {
    clear_error();
    if (!w || !t) return fail(SLLM_E_INVAL, "writer and tensor must be non-NULL");
    if (w->error != SLLM_OK) return fail(w->error, "writer already failed");
    SLLM_TRY(check_tensor_meta(t->name, t->dtype, t->ndim, t->shape, t->nbytes));
    if (t->nbytes && !t->data) return fail(SLLM_E_INVAL, "tensor '%s': data is NULL", t->name);
    if (!w->names.insert(t->name).second) return fail(SLLM_E_INVAL, "duplicate tensor name '%s'", t->name);
    uint64_t off, end;
    if (!align_up(w->cursor, w->alignment, &off) || !add_ok(off, t->nbytes, &end)) {
        w->error = SLLM_E_INVAL;
        return fail(SLLM_E_INVAL, "partition size overflows 64 bits");
    }
    int32_t st = append_zeros(w, off - w->cursor);
    if (st == SLLM_OK) st = append(w, t->data, t->nbytes);
    if (st != SLLM_OK) {
        w->error = st;
        return st;
    }
    TensorRec r;
    w->ix.set_name(r, t->name, std::strlen(t->name));
    r.dtype = t->dtype;
    r.ndim = t->ndim;
    for (uint32_t d = 0; d < t->ndim; ++d) r.shape[d] = t->shape[d];
    r.offset = off;
    r.nbytes = t->nbytes;
    w->ix.tensors.push_back(r);
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_writer_close(sllm_writer* w) try {
    Range range_("sllm_writer_close");
    clear_error();
    if (!w) return fail(SLLM_E_INVAL, "writer is NULL");
    int32_t st = w->error;
    if (st != SLLM_OK) {
        destroy(w, true);
        return fail(st, "writer failed earlier; partial files removed");
    }
    IndexData& ix = w->ix;
    ix.alignment = w->alignment;
    ix.chunk_size = w->chunk_size;
    // T: the end of the last padded slot; F: T rounded up to whole 4 KiB blocks
    if (!align_up(w->cursor, w->alignment, &ix.total) || !align_up(ix.total, kFileBlock, &ix.file_bytes)) {
        destroy(w, true);
        return fail(SLLM_E_INVAL, "partition size overflows 64 bits");
    }
    st = append_zeros(w, ix.file_bytes - w->cursor);
    if (st == SLLM_OK) st = flush(w);
    if (st == SLLM_OK && (w->flags & SLLM_CONVERT_FSYNC) && ::fsync(w->fd) != 0)
        st = fail(SLLM_E_IO, "fsync %s: %s", w->data_path.c_str(), std::strerror(errno));
    if (st == SLLM_OK && ::close(w->fd) != 0) st = fail(SLLM_E_IO, "close %s: %s", w->data_path.c_str(), std::strerror(errno));
    w->fd = -1;
    if (st == SLLM_OK) st = write_file(w->index_path, encode_index(ix), (w->flags & SLLM_CONVERT_FSYNC) != 0);
    destroy(w, st != SLLM_OK);
    return st;
} SLLM_CATCH_ALL

extern "C" void sllm_writer_abort(sllm_writer* w) {
    if (w) destroy(w, true);
}

extern "C" int32_t sllm_convert(const sllm_src_tensor* tensors, uint64_t n, const char* out_dir,
                                const sllm_convert_opts* opts) try {
    Range range_("sllm_convert");
    clear_error();
    if (n && !tensors) return fail(SLLM_E_INVAL, "tensors is NULL");
    sllm_writer* w = nullptr;
    SLLM_TRY(sllm_writer_open(out_dir, opts, &w));
    for (uint64_t i = 0; i < n; ++i) {
        int32_t st = sllm_writer_add(w, &tensors[i]);
        if (st != SLLM_OK) {
            std::string msg = sllm_last_error();
            sllm_writer_abort(w);
            return fail(st, "%s", msg.c_str());
        }
    }
    return sllm_writer_close(w);
} SLLM_CATCH_ALL
