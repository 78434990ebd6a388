"""CPU oracle for the TerMeZO step -- test infrastructure only (tests, smoke
check and the bench's CPU baseline); never imported by the product path."""
