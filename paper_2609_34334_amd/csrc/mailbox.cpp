// Cross-process mailboxes in POSIX shared memory: the CPU-based
// cross-process synchronisation of the paper's intra-node executor
// (Zero-SM Point-to-Point Executor), which coordinates the processes that
// share buffers through IPC handles.
//
// A mailbox is one shared mapping holding a fixed number of slots.  A slot
// is a 32-bit sequence word, a payload length and `slot_bytes` of payload.
// Posting writes the payload, then publishes the sequence number with a
// release store; a waiter loads the word with acquire ordering, so once it
// sees the number the payload is visible.  A waiter spins briefly, then
// sleeps on the word with a shared (not process-private) futex; a poster
// wakes sleepers only when the slot's waiter count says there are some.
// Sequence numbers compare modulo 2^32, so they may wrap.
#include <fcntl.h>
#include <linux/futex.h>
#include <sys/mman.h>
#include <sys/stat.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <chrono>
#include <climits>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <ctime>

#include "../../include/hoccl.h"
#include "errors.h"

namespace {

constexpr uint32_t kMagic = 0x484f4d42;  // "HOMB"
constexpr size_t kAlign = 64;
constexpr unsigned kMaxSlots = 1u << 20;
constexpr size_t kMaxSlotBytes = (size_t)1 << 20;
constexpr int kSpins = 2000;  // about 20 to 60 microseconds of polling

struct Header {
    uint32_t magic;
    uint32_t slots;
    uint64_t slot_bytes;
    uint64_t stride;
};

struct SlotHead {
    uint32_t seq;      // futex word
    uint32_t waiters;  // processes sleeping (or about to) on seq
    uint64_t len;
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool seq_reached(uint32_t now, uint32_t want) { return (int32_t)(now - want) >= 0; }

long futex(uint32_t *addr, int op, uint32_t val, const struct timespec *ts) {
    return syscall(SYS_futex, addr, op, val, ts, nullptr, 0);
}

bool valid_name(const char *name) {
    if (!name || name[0] != '/') return false;
    const size_t n = strnlen(name, NAME_MAX + 1);
    return n > 1 && n <= NAME_MAX && !strchr(name + 1, '/');
}

__attribute__((format(printf, 2, 3))) hoccl_status_t fail(hoccl_status_t st, const char *fmt, ...) {
    char buf[256];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    hoccl::set_error_message(buf);
    return st;
}

}  // namespace

struct hoccl_mailbox {
    char *base;
    size_t bytes;
    Header *head;
    SlotHead *slot(unsigned i) const {
        return (SlotHead *)(base + kAlign + (size_t)i * head->stride);
    }
    char *payload(unsigned i) const { return (char *)slot(i) + kAlign; }
};

extern "C" {

hoccl_status_t hoccl_mailbox_create(const char *name, unsigned slots, size_t slot_bytes,
                                    hoccl_mailbox_t **box) {
    if (!box || !valid_name(name) || slots == 0 || slots > kMaxSlots || slot_bytes > kMaxSlotBytes)
        return fail(HOCCL_ERR_INVALID_ARG, "mailbox_create: bad name, slot count or slot size");
    *box = nullptr;
    const size_t stride = kAlign + round_up(slot_bytes, kAlign);
    const size_t bytes = kAlign + (size_t)slots * stride;
    const int fd = shm_open(name, O_RDWR | O_CREAT | O_EXCL, 0600);
    if (fd < 0) return fail(HOCCL_ERR_INVALID_ARG, "shm_open(%s) failed: errno %d", name, errno);
    if (ftruncate(fd, (off_t)bytes) != 0) {
        const int e = errno;
        close(fd);
        shm_unlink(name);
        return fail(HOCCL_ERR_NO_MEMORY, "ftruncate of mailbox %s failed: errno %d", name, e);
    }
    void *p = mmap(nullptr, bytes, PROT_READ | PROT_WRITE, MAP_SHARED, fd, 0);
    close(fd);
    if (p == MAP_FAILED) {
        shm_unlink(name);
        return fail(HOCCL_ERR_NO_MEMORY, "mmap of mailbox %s failed: errno %d", name, errno);
    }
    auto *b = new hoccl_mailbox{(char *)p, bytes, (Header *)p};
    b->head->slots = slots;
    b->head->slot_bytes = slot_bytes;
    b->head->stride = stride;
    __atomic_store_n(&b->head->magic, kMagic, __ATOMIC_RELEASE);  // the pages start zeroed
    *box = b;
    return HOCCL_OK;
}

hoccl_status_t hoccl_mailbox_open(const char *name, hoccl_mailbox_t **box) {
    if (!box || !valid_name(name)) return fail(HOCCL_ERR_INVALID_ARG, "mailbox_open: bad name");
    *box = nullptr;
    const int fd = shm_open(name, O_RDWR, 0);
    if (fd < 0) return fail(HOCCL_ERR_INVALID_ARG, "shm_open(%s) failed: errno %d", name, errno);
    struct stat st;
    if (fstat(fd, &st) != 0 || (size_t)st.st_size < kAlign) {
        close(fd);
        return fail(HOCCL_ERR_INVALID_ARG, "mailbox %s is too small or unreadable", name);
    }
    const size_t bytes = (size_t)st.st_size;
    void *p = mmap(nullptr, bytes, PROT_READ | PROT_WRITE, MAP_SHARED, fd, 0);
    close(fd);
    if (p == MAP_FAILED) return fail(HOCCL_ERR_NO_MEMORY, "mmap of mailbox %s failed: errno %d", name, errno);
    auto *h = (Header *)p;
    const size_t stride = kAlign + round_up(h->slot_bytes, kAlign);
    if (__atomic_load_n(&h->magic, __ATOMIC_ACQUIRE) != kMagic || h->slots == 0 ||
        h->slots > kMaxSlots || h->slot_bytes > kMaxSlotBytes || h->stride != stride ||
        kAlign + (size_t)h->slots * stride > bytes) {
        munmap(p, bytes);
        return fail(HOCCL_ERR_INVALID_ARG, "%s is not a mailbox", name);
    }
    *box = new hoccl_mailbox{(char *)p, bytes, h};
    return HOCCL_OK;
}

hoccl_status_t hoccl_mailbox_unlink(const char *name) {
    if (!valid_name(name)) return fail(HOCCL_ERR_INVALID_ARG, "mailbox_unlink: bad name");
    if (shm_unlink(name) != 0) return fail(HOCCL_ERR_INVALID_ARG, "shm_unlink(%s) failed: errno %d", name, errno);
    return HOCCL_OK;
}

hoccl_status_t hoccl_mailbox_close(hoccl_mailbox_t *box) {
    if (!box) return HOCCL_OK;
    munmap(box->base, box->bytes);
    delete box;
    return HOCCL_OK;
}

hoccl_status_t hoccl_mailbox_post(hoccl_mailbox_t *box, unsigned slot, unsigned seq,
                                  const void *data, size_t len) {
    if (!box || slot >= box->head->slots || len > box->head->slot_bytes || (len && !data))
        return fail(HOCCL_ERR_INVALID_ARG, "mailbox_post: bad slot or payload");
    SlotHead *s = box->slot(slot);
    if (len) memcpy(box->payload(slot), data, len);
    s->len = len;
    __atomic_store_n(&s->seq, (uint32_t)seq, __ATOMIC_SEQ_CST);
    // Sequentially consistent with the waiter's increment-then-check, so a
    // sleeper either sees the new number or is counted here.
    if (__atomic_load_n(&s->waiters, __ATOMIC_SEQ_CST) != 0)
        futex(&s->seq, FUTEX_WAKE, INT_MAX, nullptr);
    return HOCCL_OK;
}

hoccl_status_t hoccl_mailbox_wait(hoccl_mailbox_t *box, unsigned slot, unsigned seq,
                                  unsigned timeout_ms) {
    if (!box || slot >= box->head->slots) return fail(HOCCL_ERR_INVALID_ARG, "mailbox_wait: bad slot");
    SlotHead *s = box->slot(slot);
    if (timeout_ms == 0)  // a poll: one look, no waiting
        return seq_reached(__atomic_load_n(&s->seq, __ATOMIC_ACQUIRE), seq) ? HOCCL_OK : HOCCL_ERR_TIMEOUT;
    for (int i = 0; i < kSpins; ++i) {
        if (seq_reached(__atomic_load_n(&s->seq, __ATOMIC_ACQUIRE), seq)) return HOCCL_OK;
        __builtin_ia32_pause();
    }
    using clock = std::chrono::steady_clock;
    const auto deadline = clock::now() + std::chrono::milliseconds(timeout_ms);
    for (;;) {
        const auto left = std::chrono::duration_cast<std::chrono::nanoseconds>(deadline - clock::now());
        if (left.count() <= 0)
            return fail(HOCCL_ERR_TIMEOUT, "mailbox_wait: slot %u did not reach %u within %u ms",
                        slot, seq, timeout_ms);
        // Sleep at most 10 ms at a time, so the deadline is re-checked even
        // if a wake-up were missed.
        const long ns = std::min<long>(left.count(), 10L * 1000 * 1000);
        __atomic_fetch_add(&s->waiters, 1u, __ATOMIC_SEQ_CST);
        const uint32_t now = __atomic_load_n(&s->seq, __ATOMIC_SEQ_CST);
        if (!seq_reached(now, seq)) {
            struct timespec ts = {0, ns};
            futex(&s->seq, FUTEX_WAIT, now, &ts);
        }
        __atomic_fetch_sub(&s->waiters, 1u, __ATOMIC_SEQ_CST);
        if (seq_reached(__atomic_load_n(&s->seq, __ATOMIC_ACQUIRE), seq)) return HOCCL_OK;
    }
}

hoccl_status_t hoccl_mailbox_read(hoccl_mailbox_t *box, unsigned slot, void *buf, size_t cap,
                                  size_t *len) {
    if (!box || slot >= box->head->slots || !len || (cap && !buf))
        return fail(HOCCL_ERR_INVALID_ARG, "mailbox_read: bad slot or buffer");
    SlotHead *s = box->slot(slot);
    const size_t n = s->len;
    *len = n;
    if (n > box->head->slot_bytes) return fail(HOCCL_ERR_INTERNAL, "mailbox_read: corrupt length");
    if (n > cap) return fail(HOCCL_ERR_INVALID_ARG, "mailbox_read: buffer too small");
    if (n) memcpy(buf, box->payload(slot), n);
    return HOCCL_OK;
}

}  // extern "C"
