"""MI355X-native gauge-coded KV-cache codec (Codec-Gauge hot path).

The codec itself is the HIP library ``libcodecgauge.so`` behind the C ABI declared in
``include/codec_gauge.h``; :mod:`paper_2607_20538_amd.codec` is its thin ctypes binding.
:mod:`paper_2607_20538_amd.synth` draws the seeded synthetic KV inputs.  Importing the
package loads nothing; the binding loads the library on first use.
"""
__all__ = ["codec", "synth"]
