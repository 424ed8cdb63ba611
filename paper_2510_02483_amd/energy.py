"""GPU energy over a timed region, from the device's accumulated-energy
counter (amd-smi), for energy per token: the report states training energy
as GPU power times time per amount of tokens (Section 3, Tables 5 and 6, in
MWh per 500 billion tokens).

Measurement only: nothing of the computed path lives here.  When the counter
cannot be read (no amd-smi, no permission, no device matching torch's current
GPU), every reading is None.
"""
from __future__ import annotations

import time


def _bdf_of_current_gpu():
    import torch

    p = torch.cuda.get_device_properties(torch.cuda.current_device())
    dom, bus, dev = getattr(p, "pci_domain_id", None), getattr(p, "pci_bus_id", None), getattr(p, "pci_device_id", None)
    if bus is None or dev is None:
        return None
    return (int(dom or 0), int(bus), int(dev))


class EnergyMeter:
    """Reads the accumulated energy (joules) of the GPU torch is using."""

    def __init__(self):
        self.handle = None
        self.error = None
        try:
            import amdsmi

            self._smi = amdsmi
            amdsmi.amdsmi_init()
            handles = amdsmi.amdsmi_get_processor_handles()
            want = _bdf_of_current_gpu()
            for h in handles:
                bdf = amdsmi.amdsmi_get_gpu_device_bdf(h)  # "dddd:bb:dd.f"
                dom, bus, rest = bdf.split(":")
                key = (int(dom, 16), int(bus, 16), int(rest.split(".")[0], 16))
                if want is None and len(handles) == 1 or key == want:
                    self.handle = h
                    break
            if self.handle is None:
                self.error = f"no amd-smi device matches the current GPU {want}"
            else:
                self.joules()
        except Exception as e:  # noqa: BLE001  (any failure: report no energy)
            self.handle = None
            self.error = f"{type(e).__name__}: {e}"

    def joules(self):
        if self.handle is None:
            return None
        e = self._smi.amdsmi_get_energy_count(self.handle)
        return e["energy_accumulator"] * e["counter_resolution"] * 1e-6

    def gfx_clocks(self):
        """Current shader clock of each XCD in MHz (the firmware's metrics
        table), or None when it cannot be read."""
        if self.handle is None:
            return None
        try:
            m = self._smi.amdsmi_get_gpu_metrics_info(self.handle)
        except Exception:  # noqa: BLE001
            return None
        v = m.get("current_gfxclks")
        if not isinstance(v, (list, tuple)):
            v = [m.get("current_gfxclk")]
        return v

    def measure(self, fn, min_seconds: float = 2.0):
        """Run fn() (which must synchronise the device at its end) repeatedly
        for at least min_seconds; return (calls, seconds, joules or None,
        mean shader clock in MHz or None).  The clock is sampled every 10 ms
        by a second thread while the loop runs."""
        import threading

        samples, stop = [], threading.Event()

        def sample():
            while not stop.wait(0.01):
                c = self.gfx_clocks()
                if c is not None:
                    samples.append(c)

        th = threading.Thread(target=sample, daemon=True) if self.handle is not None else None
        e0 = self.joules()
        t0 = time.perf_counter()
        if th is not None:
            th.start()
        calls = 0
        while True:
            fn()
            calls += 1
            dt = time.perf_counter() - t0
            if dt >= min_seconds:
                break
        if th is not None:
            stop.set()
            th.join()
        e1 = self.joules()
        return calls, dt, (None if e0 is None or e1 is None else e1 - e0), mean_clock_mhz(samples)


def mean_clock_mhz(samples):
    """Mean shader clock (MHz) over clock samples, each a list of per-XCD
    readings; readings that are not numbers in the chip's range (the metrics
    table marks missing values with "N/A" or 0xFFFF) are left out.  None
    when no reading is valid."""
    vals = [float(v) for smp in samples for v in smp
            if isinstance(v, (int, float)) and not isinstance(v, bool) and 0 < v < 10000]
    return round(sum(vals) / len(vals), 1) if vals else None


def report(calls: int, seconds: float, joules, tokens_per_call: int) -> dict:
    """Energy figures of a measured loop (None values when no energy reading)."""
    out = {"calls": calls, "seconds": round(seconds, 3)}
    if joules is None or joules <= 0:
        out.update(joules=None, avg_power_w=None, joules_per_token=None, mwh_per_500b_tokens=None)
        return out
    jpt = joules / (calls * tokens_per_call)
    out.update(joules=round(joules, 2), avg_power_w=round(joules / seconds, 1), joules_per_token=jpt,
               mwh_per_500b_tokens=round(jpt * 500e9 / 3.6e9, 4))
    return out
