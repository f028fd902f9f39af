"""Co-location profile and the smallest-safe-share table (Section 3.4, dynamic
SM partitioning).

The encode worker may share its GPU with a local prefill worker on disjoint
compute-unit subsets, re-split at every micro-batch.  Encode latency is
profiled at a few allocation levels (five: 10, 30, 50, 70 and 90% of the
device) across batch sizes; for every level the table keeps the largest batch
size whose latency stays within 20% of the exclusive-access latency (the
threshold of the paper's latency-versus-allocation figure).  At run time encode
takes the smallest level whose table entry covers the current micro-batch;
a batch no level covers runs with the whole device.

The share is taken on MI355X by occupancy (``eas_cu_reserve``, include/
eas_colocate.h): a reservation holds whole compute units, so the encoder's
kernels run on the rest.  The reservation needs a hardware queue of its own:
HIP maps streams onto a few hardware queues per process (4 by default), and
streams that share one run in order, so encode work placed behind a
reservation would wait for it.  A profiling process therefore keeps its
streams few (one reservation stream and one measuring stream, made once) and
starts with ``GPU_MAX_HW_QUEUES`` raised (16).  The lowest level is 12.5% instead of 10%: 32 CUs, one
for each of the device's 32 shader engines.  With fewer, some shader engine has
no free CU, and the encoder's kernels wait behind it until the reservation
ends (measured: 26 free CUs stall the encoder for the whole reservation, 32 do
not).
"""
import ctypes
import statistics
import time

from .eas import LIB, EAS_OK, EasError

EXPORTS = ("eas_cu_reserve", "eas_cu_reserve_max")
LIB.eas_cu_reserve.argtypes = [ctypes.c_int32, ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
LIB.eas_cu_reserve.restype = ctypes.c_int32
LIB.eas_cu_reserve_max.argtypes = [ctypes.c_int32]
LIB.eas_cu_reserve_max.restype = ctypes.c_int32


def reserve_max(device_cus):
    """Largest share eas_cu_reserve accepts: all but one CU per shader engine."""
    return int(LIB.eas_cu_reserve_max(int(device_cus)))

LEVELS = (0.125, 0.3, 0.5, 0.7, 0.9)   # allocation levels profiled (fractions of the device's CUs)
THRESHOLD = 0.2                      # latency within 20% of exclusive access counts as safe


def device_cus():
    import torch
    return torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count


_streams = {}


def _stream(role):
    """A stream made once per process for ``role`` ("reserve", "measure")."""
    import torch
    if role not in _streams:
        _streams[role] = torch.cuda.Stream()
    return _streams[role]


class CuReservation:
    """Holds ``n_cus`` compute units from ``__enter__`` (once every workgroup is
    resident) until ``__exit__``, or until ``max_s`` seconds have passed."""

    def __init__(self, n_cus, max_s=10.0, start_timeout_s=5.0):
        self.n, self.max_s, self.timeout = int(n_cus), float(max_s), float(start_timeout_s)

    def __enter__(self):
        import torch
        self.started = torch.zeros(self.n, dtype=torch.int32, pin_memory=True)
        self.release = torch.zeros(1, dtype=torch.int32, pin_memory=True)
        self.stream = _stream("reserve")
        t_sync = time.time()
        torch.cuda.synchronize()   # an idle device: every workgroup finds a free CU
        self.t_launch = time.time()
        self.sync_s = self.t_launch - t_sync
        st = LIB.eas_cu_reserve(self.n, self.max_s, self.started.data_ptr(), self.release.data_ptr(),
                                self.stream.cuda_stream)
        if st != EAS_OK:
            raise EasError(st, "eas_cu_reserve")
        t0 = time.time()
        while int(self.started.sum()) < self.n:
            if time.time() - t0 > self.timeout:
                self._end()
                raise RuntimeError("%d of %d reserving workgroups resident after %.1f s"
                                   % (int(self.started.sum()), self.n, self.timeout))
            time.sleep(1e-4)
        self.ready_s = time.time() - self.t_launch   # from the launch until every block is resident
        return self

    def _end(self):
        t0 = time.time()
        self.held_s = t0 - self.t_launch   # from the launch to the release
        self.release[0] = 1
        self.stream.synchronize()
        self.release_s = time.time() - t0   # from the release to the reservation's end

    def lapsed(self):
        """True when the reservation may have ended (time limit) before its release."""
        return self.held_s >= 0.9 * self.max_s

    def __exit__(self, *exc):
        self._end()
        return False


def encode_latency_ms(run, share, reps=3, cus=None, max_s=10.0, log=None):
    """Median time (ms) of ``run(stream)`` -- one micro-batch on a torch stream --
    with the encoder limited to ``share`` of the CUs (1.0: exclusive access);
    None when a reservation came close to its time limit before it was released
    (the encoder stalled behind it, or the share lapsed while it ran).  ``log``: optional callable given one line per
    repetition."""
    import torch
    cus = cus or device_cus()
    hold = int(round((1.0 - share) * cus))
    stream = _stream("measure")
    times, lapsed = [], False
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

        def timed():
            e0.record(stream)
            run(stream)
            e1.record(stream)
            e1.synchronize()

        w0 = time.time()
        if hold > 0:
            with CuReservation(hold, max_s) as r:
                timed()
        else:
            r = None
            torch.cuda.synchronize()
            timed()
        times.append(e0.elapsed_time(e1))
        lapsed = lapsed or (r is not None and r.lapsed())
        if log:
            log("share %.2f (%d CUs held): %.3f ms encode, %.3f s in all; %s" % (
                share, hold, times[-1], time.time() - w0,
                "sync %.3f s, resident after %.3f s, held %.3f s, released in %.3f s%s" % (
                    r.sync_s, r.ready_s, r.held_s, r.release_s, " (lapsed)" if r.lapsed() else "")
                if r else "no reservation"))
    if lapsed:
        return None
    return statistics.median(times)


def profile(run_for_batch, batches, levels=LEVELS, reps=3, max_s=10.0, log=None):
    """Encode latency (ms) per batch size, exclusive and at every level.
    ``run_for_batch(b)`` returns a callable running one micro-batch of b on a
    given stream."""
    exclusive, latency = {}, {lv: {} for lv in levels}
    for b in batches:
        blog = (lambda m, b=b: log("micro-batch %d, %s" % (b, m))) if log else None
        run = run_for_batch(b)
        encode_latency_ms(run, 1.0, reps=1)   # warm-up
        exclusive[b] = encode_latency_ms(run, 1.0, reps, max_s=max_s, log=blog)
        for lv in levels:
            latency[lv][b] = encode_latency_ms(run, lv, reps, max_s=max_s, log=blog)
    return exclusive, latency


def safe_share_table(latency, exclusive, threshold=THRESHOLD):
    """Level -> the largest profiled batch size whose latency at that level is
    within ``threshold`` of its exclusive-access latency (0: none; an
    unmeasured latency, None, never qualifies)."""
    return {lv: max([b for b, ms in row.items() if ms is not None and ms <= (1.0 + threshold) * exclusive[b]],
                    default=0)
            for lv, row in latency.items()}


def select_share(table, batch):
    """The smallest level whose entry covers ``batch``; 1.0 (the whole device)
    when none does."""
    fits = [lv for lv, b in table.items() if b >= batch]
    return min(fits) if fits else 1.0
