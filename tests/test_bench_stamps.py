"""Host checks of bench.py's phase-stamp analysis (stamp_summary, attend_step_waves) on
synthetic records whose answers are known by construction: the figures of
profiles/phase_timelines_wan.md come from these two functions."""
import numpy as np

import bench

WG, WAVES, POINTS = 2048, 8, 16


def _rec():
    return np.zeros((WG, WAVES, POINTS), dtype=np.uint64)


def test_stamp_summary_takes_the_last_wave_and_the_workgroup_start():
    rec = _rec()
    # three live workgroups; ticks of 10 ns. Workgroup w starts at 1000 + 10 w (wave 0 first).
    for w in range(3):
        s = 1000 + 10 * w
        for v in range(4):
            rec[w, v, 0] = s + v          # later waves start a tick apart
            rec[w, v, 1] = s + 100 + v    # point 1: the last wave at +103
            rec[w, v, 2] = s + 300 + 2 * w  # point 2: +300, +302, +304
    out = bench.stamp_summary(rec, {0: "start", 1: "one", 2: "two", 5: "never reached"})
    assert out["workgroups"] == 3
    assert out["points_us"] == {"one": 1.03, "two": 3.02}  # medians, in us
    assert out["workgroup_us_median"] == 3.02 and out["workgroup_us_max"] == 3.04
    assert out["start_spread_us"] == 0.2
    assert out["span_us"] == round((1020 + 304 - 1000) / 100, 2)


def test_attend_step_waves_separates_older_and_younger_waves():
    rec = _rec()
    # one workgroup; step i releases at 1000 + 150 i ticks. Older waves (0-3) end their stream
    # 30 ticks before the release, younger ones (4-7) 5 ticks before; SIMD s ends 1 tick later
    # than SIMD s - 1 (so the SIMDs end 3 ticks apart).
    rec[0, :, 0] = 1
    for i in range(4):
        release = 1000 + 150 * i
        for v in range(8):
            simd = v % 4
            end = release - (30 if v < 4 else 5) + simd - 3
            rec[0, v, 2 + 2 * i] = end
            rec[0, v, 3 + 2 * i] = release
    out = bench.attend_step_waves(rec)
    assert out["step_us_median"] == 1.5
    # waits: older 30 - (simd - 3) = 30..33 ticks, median 31.5; younger 5..8, median 6.5
    assert out["older_wave_barrier_wait_us_median"] == 0.315
    assert out["younger_wave_barrier_wait_us_median"] == 0.065
    assert out["older_wave_ends_first_fraction"] == 1.0
    assert out["one_wave_alone_us_median"] == 0.25
    assert out["last_stream_end_to_release_us_median"] == 0.05
    assert out["simd_end_spread_us_median"] == 0.03
    assert out["samples"] == 16


def test_attend_segments_splits_the_switch_and_compares_segment_counts():
    rec = _rec()
    # workgroup 0: one segment, 1000 ticks; workgroups 1 and 2: two segments, 1200 and 1220
    for w, (dur, two) in enumerate(((1000, False), (1200, True), (1220, True))):
        rec[w, :, 0] = 10
        rec[w, :, 10] = 10 + dur - 50     # last step done, 50 ticks before the stores are done
        rec[w, :, 11] = 10 + dur
        if two:
            rec[w, :, 12] = 400           # first segment's last step
            rec[w, :, 13] = 400 + 60 + 2 * w  # its partial results issued
            rec[w, :, 14] = 400 + 110     # the second segment's first tiles landed
    out = bench.attend_segments(rec)
    assert out["two_segment_workgroups"] == 2
    assert out["switch_us_median"] == 1.1
    assert out["switch_stores_issued_us_median"] == 0.63
    assert out["switch_to_tiles_landed_us_median"] == 0.47
    assert out["end_tail_us_median"] == 0.5
    assert out["one_segment_workgroup_us_median"] == 10.0
    assert out["two_segment_workgroup_us_median"] == 12.1
