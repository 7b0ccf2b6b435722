"""GPU clock and power during a measured interval, read in process.

The paper's control plane rests on measured clock, power and throughput per
serving phase (§III-B Observation 2; App. B.3's power and latency models).
This module reads them for one GPU through the amdsmi library (no subprocess):
a sampler thread polls the GPU metrics table (current GFX clock, current
socket power) every few milliseconds while a leg runs; the energy
accumulator's reading is kept beside it. Read-only: nothing here
changes a clock, a power cap or any other device setting.

Use:
    tel = Telemetry()                 # binds to the GPU torch calls cuda:0
    with tel.leg() as rec:
        ... launch and synchronise ...
    rec.result  # {"gfxclk_mhz": {...}, "power_w": {...}, ...}
    tel.observe(run, sync)            # the same over a replay window long
                                      # enough for the driver's refresh rate
When amdsmi is missing or refuses (no driver access), every result is
{"available": False, "reason": ...} and measurements proceed without it.

From the command line, `python -m paper_2608_21719_amd.telemetry -- CMD ...`
runs CMD as a child process (GPU 0) and prints its output followed by the
clock and power sampled while it ran, as one JSON line.
"""
import threading
import time


def _bdf_of_torch_device(index: int):
    try:
        import torch
        p = torch.cuda.get_device_properties(index)
        return (int(p.pci_domain_id), int(p.pci_bus_id), int(p.pci_device_id))
    except Exception:
        return None


class _Leg:
    def __init__(self, tel, period_s):
        self.tel = tel
        self.period_s = period_s
        self.result = None
        self._clk, self._pw = [], []
        self._stop = threading.Event()

    def _sample(self):
        smi, h = self.tel.smi, self.tel.handle
        while not self._stop.is_set():
            try:
                m = smi.amdsmi_get_gpu_metrics_info(h)
                clk, pw = m.get("current_gfxclk"), m.get("current_socket_power")
                if isinstance(clk, (int, float)) and clk > 0:
                    self._clk.append(float(clk))
                if isinstance(pw, (int, float)) and pw > 0:
                    self._pw.append(float(pw))
            except Exception:
                pass
            self._stop.wait(self.period_s)

    def __enter__(self):
        if not self.tel.available:
            self.result = {"available": False, "reason": self.tel.reason}
            return self
        self._e0 = self.tel.energy_j()
        self._t0 = time.perf_counter()
        self._th = threading.Thread(target=self._sample, daemon=True)
        self._th.start()
        return self

    def __exit__(self, *exc):
        if not self.tel.available:
            return False
        self._stop.set()
        self._th.join()
        dt = time.perf_counter() - self._t0
        e1 = self.tel.energy_j()
        res = {"available": True, "seconds": dt, "samples": len(self._clk)}

        def stats(v):
            if not v:
                return None
            v = sorted(v)
            return {"mean": sum(v) / len(v), "min": v[0], "median": v[len(v) // 2], "max": v[-1]}

        res["gfxclk_mhz"] = stats(self._clk)
        res["power_w"] = stats(self._pw)
        if self._e0 is not None and e1 is not None and dt > 0:
            # raw energy-counter reading; on MI355X it agrees with the sampled
            # socket power at idle but reads about 1.3x it under load, so the
            # sampled power is the figure to use
            res["energy_counter_j"] = e1 - self._e0
            res["energy_counter_mean_w"] = (e1 - self._e0) / dt
        self.result = res
        return False


class Telemetry:
    def __init__(self, torch_device: int = 0):
        self.available = False
        self.reason = ""
        self.smi = None
        self.handle = None
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            handles = amdsmi.amdsmi_get_processor_handles()
            if not handles:
                raise RuntimeError("amdsmi lists no GPU")
            want = _bdf_of_torch_device(torch_device)
            self.handle = handles[0]
            if want is not None and len(handles) > 1:
                for h in handles:
                    try:
                        b = amdsmi.amdsmi_get_gpu_device_bdf(h)  # "dddd:bb:dd.f"
                        dom, bus, dev = b.split(":")[0], b.split(":")[1], b.split(":")[2].split(".")[0]
                        if (int(dom, 16), int(bus, 16), int(dev, 16)) == want:
                            self.handle = h
                            break
                    except Exception:
                        continue
            self.smi = amdsmi
            self.available = True
        except Exception as e:  # no library, no driver access: measure without telemetry
            self.reason = f"{type(e).__name__}: {e}"

    def energy_j(self):
        try:
            r = self.smi.amdsmi_get_energy_count(self.handle)
            return r["energy_accumulator"] * r["counter_resolution"] * 1e-6  # resolution is in microjoules
        except Exception:
            return None

    def static_info(self) -> dict:
        """Clock range and power cap as the driver reports them (read-only)."""
        if not self.available:
            return {"available": False, "reason": self.reason}
        out = {"available": True}
        try:
            ci = self.smi.amdsmi_get_clock_info(self.handle, self.smi.AmdSmiClkType.SYS)
            out["gfxclk_min_mhz"], out["gfxclk_max_mhz"] = ci.get("min_clk"), ci.get("max_clk")
        except Exception as e:
            out["clock_info_error"] = str(e)
        try:
            pc = self.smi.amdsmi_get_power_cap_info(self.handle)
            out["power_cap_w"] = pc.get("power_cap", 0) / 1e6 if pc.get("power_cap", 0) > 1e5 else pc.get("power_cap")
        except Exception as e:
            out["power_cap_error"] = str(e)
        return out

    def leg(self, period_s: float = 0.005) -> _Leg:
        return _Leg(self, period_s)

    def observe(self, run, sync, seconds: float = 1.5, settle_s: float = 0.4) -> dict:
        """Clock and power while `run` repeats: the driver's metrics table and
        energy counter refresh every few tens of milliseconds, too slowly for
        a short timed region, so the same work is replayed for `seconds`
        after `settle_s` of warm-up (clock and power ramp after a change of
        load) and observed over that window."""
        import time as _t
        t0 = _t.perf_counter()
        n = 0
        while _t.perf_counter() - t0 < settle_s:
            run()
            sync()
            n += 1
        # batches of about 20 ms between synchronisations keep the GPU busy
        batch = max(1, int(0.02 / ((_t.perf_counter() - t0) / n)))
        with self.leg() as rec:
            t0 = _t.perf_counter()
            while _t.perf_counter() - t0 < seconds:
                for _ in range(batch):
                    run()
                sync()
        return rec.result


def main(argv=None) -> int:
    """Run a command as a child process and report GPU 0's clock and power
    over its run (the child owns its own GPU work; nothing is exec'd)."""
    import json
    import subprocess
    import sys
    args = list(sys.argv[1:] if argv is None else argv)
    if args and args[0] == "--":
        args = args[1:]
    if not args:
        print("usage: python -m paper_2608_21719_amd.telemetry -- CMD [ARGS...]", file=sys.stderr)
        return 2
    tel = Telemetry(0)
    with tel.leg() as rec:
        r = subprocess.run(args, capture_output=True, text=True)
    sys.stdout.write(r.stdout)
    sys.stderr.write(r.stderr)
    print(json.dumps({"command": args, "returncode": r.returncode, "static": tel.static_info(),
                      "telemetry": rec.result}))
    return r.returncode


if __name__ == "__main__":
    raise SystemExit(main())
