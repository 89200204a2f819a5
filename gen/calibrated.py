"""Frozen Zipf bias scales written by gen/calibrate.py."""
ZIPF_C = {2: 0.320312, 4: 0.267578}
