"""Device power telemetry: amd-smi socket power sampled on a thread.

The paper samples every device every 0.5 s and records, per sample, the
timestamp, elapsed time, device index, training phase, power, utilisation and
temperature (section 4.4); ``PowerSampler`` keeps the same record for the one
MI355X, labelling each sample with the phase the caller has set.  Samples can
also be forwarded to a listener (the occupancy monitor) as they arrive.
"""
from __future__ import annotations

import threading
import time


class PowerSampler:
    """amd-smi socket power every ``period`` seconds on a thread; ``ok`` is False when it is unavailable."""

    def __init__(self, period: float = 0.5, gpu: int = 0):
        self.period = period
        self.gpu = gpu
        self.samples = []      # (perf_counter time, watts)
        self.records = []      # telemetry records (dicts)
        self.field = None
        self.phase = "idle"
        self.listener = None   # called with each power sample in watts
        self._stop = threading.Event()
        self._thr = None
        self._t0 = None
        self.ok = False
        try:
            import amdsmi

            amdsmi.amdsmi_init()
            self._smi = amdsmi
            self._h = amdsmi.amdsmi_get_processor_handles()[gpu]
            self.ok = self.read() is not None
        except Exception:
            self.ok = False

    def read(self):
        """Socket power in watts, or None."""
        try:
            info = self._smi.amdsmi_get_power_info(self._h)
        except Exception:
            return None
        for key in ("current_socket_power", "average_socket_power", "socket_power"):
            v = info.get(key) if isinstance(info, dict) else None
            if isinstance(v, (int, float)) and v > 0:
                self.field = key
                return float(v)
        return None

    def _util_temp(self):
        util = temp = None
        try:
            util = self._smi.amdsmi_get_gpu_activity(self._h).get("gfx_activity")
        except Exception:
            pass
        try:
            temp = self._smi.amdsmi_get_temp_metric(self._h, self._smi.AmdSmiTemperatureType.HOTSPOT,
                                                    self._smi.AmdSmiTemperatureMetric.CURRENT)
        except Exception:
            pass
        return util, temp

    def _run(self):
        while not self._stop.is_set():
            t = time.perf_counter()
            p = self.read()
            if p is not None:
                self.samples.append((t, p))
                util, temp = self._util_temp()
                self.records.append({"timestamp": time.time(), "elapsed_s": round(t - self._t0, 3), "gpu": self.gpu,
                                     "phase": self.phase, "power_w": p, "gfx_util": util, "temp_c": temp})
                if self.listener is not None:
                    self.listener(p)
            self._stop.wait(self.period)

    def start(self):
        if self.ok:
            self.samples, self.records = [], []
            self._t0 = time.perf_counter()
            self._stop.clear()
            self._thr = threading.Thread(target=self._run, daemon=True)
            self._thr.start()

    def stop(self):
        if self._thr:
            self._stop.set()
            self._thr.join()
            self._thr = None
        return list(self.samples)


def energy_joules(samples, t0: float, t1: float):
    """Integrate power over [t0, t1] with a zero-order hold between samples (None without samples)."""
    if not samples:
        return None
    e = 0.0
    for i, (t, p) in enumerate(samples):
        a = max(t, t0)
        b = min(samples[i + 1][0] if i + 1 < len(samples) else t1, t1)
        if b > a:
            e += p * (b - a)
    first_t, first_p = samples[0]
    if first_t > t0:
        e += first_p * (first_t - t0)
    return e
